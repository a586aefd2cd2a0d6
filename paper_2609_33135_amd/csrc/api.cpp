// api.cpp -- the C ABI of include/mpfa.h: host-side validation (no HIP call
// before an argument set is accepted), launch configuration and the decode
// partition policy.
#include "mpfa.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "mpfa_internal.h"

static_assert(MPFA_STATIC_SCRATCH_BYTES == mpfa::kStaticScratchBytes,
              "public and internal sizes of the static decode scratch must agree");

#ifdef MPFA_DEBUG_CHECKS
#include <vector>
#endif

namespace {

constexpr int kPrefillRows = 256;   // query rows per prefill workgroup
constexpr int kMaxKvHeads = mpfa::kMaxKvHeadsQuant;
constexpr int kMaxDecodeGroup = 8;  // query heads per KV head packed in one decode wave
constexpr float kLambda = 0.12751743074173085f;   // log2(e) / sqrt(128)

bool heads_ok(int h_q, int h_kv) {
  return h_q >= 1 && h_kv >= 1 && h_q <= MPFA_MAX_HEADS && h_kv <= kMaxKvHeads && h_q % h_kv == 0;
}

// partition counters of the fused step follow the decode states, 256-byte aligned
size_t mixed_counter_offset(size_t state_bytes) { return (state_bytes + 255) / 256 * 256; }

#ifdef MPFA_DEBUG_CHECKS
// ---- data checks of the debug library: index arrays copied to the host after
// the stream's earlier work, inputs scanned for non-finite values on the device
template <typename T>
bool to_host(const T* dev, size_t n, std::vector<T>& out) {
  out.resize(n);
  return n == 0 || hipMemcpy(out.data(), dev, n * sizeof(T), hipMemcpyDeviceToHost) == hipSuccess;
}

mpfa_status scan_nonfinite(const void* x, int64_t n, hipStream_t s) {
  int* flag = nullptr;
  if (hipMalloc(&flag, sizeof(int)) != hipSuccess) return MPFA_ERR_HIP;
  int h = 0;
  const bool ok = hipMemsetAsync(flag, 0, sizeof(int), s) == hipSuccess &&
                  mpfa::launch_scan_nonfinite(static_cast<const uint16_t*>(x), n, flag, s) == hipSuccess &&
                  hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, s) == hipSuccess &&
                  hipStreamSynchronize(s) == hipSuccess;
  (void)hipFree(flag);
  if (!ok) return MPFA_ERR_HIP;
  return h ? MPFA_ERR_DATA : MPFA_OK;
}

// page-table entries of the pages a sequence of kv_len keys uses
bool pages_ok(const std::vector<int32_t>& pt, int b, int max_pages, int kv_len, int64_t num_pages) {
  for (int i = 0; i < (kv_len + 63) / 64; ++i) {
    const int32_t e = pt[(size_t)b * max_pages + i];
    if (e < 0 || (num_pages > 0 && e >= num_pages)) return false;
  }
  return true;
}

mpfa_status check_quant(const mpfa_quant_args* a, hipStream_t s) {
  if (hipStreamSynchronize(s) != hipSuccess) return MPFA_ERR_HIP;
  std::vector<int32_t> cu;
  std::vector<int64_t> slots;
  if (!to_host(a->cu_seqlens, (size_t)a->batch + 1, cu) || !to_host(a->slot_mapping, (size_t)a->total_tokens, slots))
    return MPFA_ERR_HIP;
  if (cu[0] != 0 || cu[a->batch] != a->total_tokens) return MPFA_ERR_DATA;
  for (int b = 0; b < a->batch; ++b)
    if (cu[b + 1] < cu[b] || cu[b + 1] - cu[b] > a->max_seqlen) return MPFA_ERR_DATA;
  for (int64_t t = 0; t < a->total_tokens; ++t)
    if (slots[t] < 0 || slots[t] >= 64 * a->num_pages) return MPFA_ERR_DATA;
  if (a->flags & MPFA_PV_NVFP4)   // fresh prefill: token i at slot i % 64 of its page
    for (int b = 0; b < a->batch; ++b)
      for (int64_t i = 0; i < cu[b + 1] - cu[b]; ++i) {
        const int64_t first = slots[cu[b] + i - i % 64];
        if (first % 64 != 0 || slots[cu[b] + i] != first + i % 64) return MPFA_ERR_DATA;
      }
  const int64_t T = a->total_tokens;
  mpfa_status st = scan_nonfinite(a->q, T * a->h_q * MPFA_HEAD_DIM, s);
  if (st == MPFA_OK) st = scan_nonfinite(a->k, T * a->h_kv * MPFA_HEAD_DIM, s);
  if (st == MPFA_OK) st = scan_nonfinite(a->v, T * a->h_kv * MPFA_HEAD_DIM, s);
  return st;
}

mpfa_status check_prefill(const mpfa_prefill_args* a, hipStream_t s) {
  if (hipStreamSynchronize(s) != hipSuccess) return MPFA_ERR_HIP;
  std::vector<int32_t> cu, qs, kv, pt;
  if (!to_host(a->cu_seqlens_q, (size_t)a->batch + 1, cu) || !to_host(a->q_start, (size_t)a->batch, qs) ||
      !to_host(a->kv_len, (size_t)a->batch, kv) || !to_host(a->page_table, (size_t)a->batch * a->max_pages, pt))
    return MPFA_ERR_HIP;
  for (int b = 0; b < a->batch; ++b) {
    const int n = cu[b + 1] - cu[b];
    if (n < 0 || n > a->max_seqlen_q || qs[b] < 0 || (int64_t)qs[b] + n > kv[b] ||
        (int64_t)kv[b] > 64LL * a->max_pages || !pages_ok(pt, b, a->max_pages, kv[b], a->num_pages))
      return MPFA_ERR_DATA;
  }
  return MPFA_OK;
}

mpfa_status check_decode(const mpfa_decode_args* a, hipStream_t s) {
  if (hipStreamSynchronize(s) != hipSuccess) return MPFA_ERR_HIP;
  std::vector<int32_t> kv, pt;
  if (!to_host(a->kv_len, (size_t)a->batch, kv) || !to_host(a->page_table, (size_t)a->batch * a->max_pages, pt))
    return MPFA_ERR_HIP;
  for (int b = 0; b < a->batch; ++b) {
    if (kv[b] < 1 || (int64_t)kv[b] > 64LL * a->max_pages ||
        (kv[b] + a->partition_tokens - 1) / a->partition_tokens > a->max_partitions ||
        !pages_ok(pt, b, a->max_pages, kv[b], a->num_pages))
      return MPFA_ERR_DATA;
  }
  return MPFA_OK;
}
#endif

}  // namespace

// Host-side validation of the prefill arguments and their launch parameters.
static mpfa_status prefill_params(const mpfa_prefill_args* a, mpfa::PrefillParams& p) {
  if (!a) return MPFA_ERR_INVALID;
  if (a->head_dim != MPFA_HEAD_DIM) return a->head_dim > 0 ? MPFA_ERR_UNSUPPORTED : MPFA_ERR_INVALID;
  if (a->batch < 1 || a->max_seqlen_q < 0 || a->max_pages < 1) return MPFA_ERR_INVALID;
  if (!heads_ok(a->h_q, a->h_kv)) return MPFA_ERR_INVALID;
  if (a->flags & ~(MPFA_SMOOTH | MPFA_SEED_MFMA | MPFA_SEED_ELEMWISE | MPFA_MXFP4 | MPFA_PV_BF16 |
                   MPFA_PV_NVFP4))
    return MPFA_ERR_INVALID;
  if ((a->flags & MPFA_SEED_MFMA) && (a->flags & MPFA_SEED_ELEMWISE)) return MPFA_ERR_INVALID;
  const uint32_t pvp = a->flags & (MPFA_PV_BF16 | MPFA_PV_NVFP4);
  if (pvp == (MPFA_PV_BF16 | MPFA_PV_NVFP4) || (pvp && !a->v_aux)) return MPFA_ERR_INVALID;
  if ((pvp & MPFA_PV_NVFP4) && a->num_pages < 1) return MPFA_ERR_INVALID;
  if (pvp && (a->flags & (MPFA_MXFP4 | MPFA_SEED_MFMA | MPFA_SEED_ELEMWISE))) return MPFA_ERR_UNSUPPORTED;
  const bool smooth = a->flags & MPFA_SMOOTH;
  if (!a->cu_seqlens_q || !a->q_start || !a->kv_len || !a->page_table || !a->q_codes ||
      !a->q_scales || !a->q_tscale || !a->k_codes || !a->k_scales || !a->v_codes ||
      !a->k_tscale || !a->out || (smooth && !a->ds))
    return MPFA_ERR_INVALID;
  const int64_t n_qtiles = ((int64_t)a->max_seqlen_q + kPrefillRows - 1) / kPrefillRows;
  if (n_qtiles * a->h_q * (int64_t)a->batch > INT32_MAX) return MPFA_ERR_INVALID;

  p = mpfa::PrefillParams{};
  p.batch = a->batch;
  p.h_q = a->h_q;
  p.h_kv = a->h_kv;
  p.max_pages = a->max_pages;
  p.n_qtiles = (int)n_qtiles;
  p.smooth = smooth;
  p.seed_mfma = (a->flags & MPFA_SEED_MFMA) != 0;
  p.seed_elem = (a->flags & MPFA_SEED_ELEMWISE) != 0;
  p.pv = (a->flags & MPFA_PV_BF16) ? 1 : (a->flags & MPFA_PV_NVFP4) ? 2 : 0;
  p.v_aux = static_cast<const uint8_t*>(a->v_aux);
  p.num_pages = a->num_pages;
  p.mx = (a->flags & MPFA_MXFP4) != 0;
  p.xcd_remap = (a->h_kv % 8) == 0;
  p.lam = kLambda;
  p.cu_seqlens_q = a->cu_seqlens_q;
  p.q_start = a->q_start;
  p.kv_len = a->kv_len;
  p.page_table = a->page_table;
  p.q_codes = a->q_codes;
  p.q_scales = a->q_scales;
  p.q_tscale = a->q_tscale;
  p.k_codes = a->k_codes;
  p.k_scales = a->k_scales;
  p.v_codes = a->v_codes;
  p.ds = static_cast<const uint16_t*>(a->ds);
  p.k_tscale = a->k_tscale;
  p.out = static_cast<uint16_t*>(a->out);
  return MPFA_OK;
}


// Host-side validation of the decode arguments and their launch parameters,
// apart from the workspace.
static mpfa_status decode_args_params(const mpfa_decode_args* a, mpfa::DecodeParams& p) {
  if (!a) return MPFA_ERR_INVALID;
  if (a->head_dim != MPFA_HEAD_DIM) return a->head_dim > 0 ? MPFA_ERR_UNSUPPORTED : MPFA_ERR_INVALID;
  if (a->batch < 1 || a->batch > 65535 || a->max_pages < 1 || a->max_partitions < 1)
    return MPFA_ERR_INVALID;
  if (a->partition_tokens < MPFA_KV_TILE || a->partition_tokens % MPFA_KV_TILE)
    return MPFA_ERR_INVALID;
  if (!heads_ok(a->h_q, a->h_kv)) return MPFA_ERR_INVALID;
  if (a->h_q / a->h_kv > kMaxDecodeGroup) return MPFA_ERR_UNSUPPORTED;
  if (a->flags & (MPFA_PV_BF16 | MPFA_PV_NVFP4)) return MPFA_ERR_UNSUPPORTED;
  if (a->flags & ~(MPFA_SMOOTH | MPFA_MXFP4)) return MPFA_ERR_INVALID;
  {
    // up to kDecodePackedMaxBatch sequences the decode grid is one dimension of 256-thread
    // workgroups: per (sequence, group of 4 partitions) pair, the KV heads
    // rounded up to 8; above, its x dimension is the odd group count
    const int64_t groups = (a->max_partitions + 3) / 4;
    const int64_t blocks = a->batch <= mpfa::kDecodePackedMaxBatch
                               ? (int64_t)a->batch * groups * ((a->h_kv + 7) / 8 * 8)
                               : (groups | 1);
    if (blocks * 256 > (int64_t)UINT32_MAX) return MPFA_ERR_UNSUPPORTED;
  }
  const bool smooth = a->flags & MPFA_SMOOTH;
  if (!a->kv_len || !a->page_table || !a->q_codes || !a->q_scales || !a->q_tscale ||
      !a->k_codes || !a->k_scales || !a->v_codes || !a->k_tscale || !a->out || (smooth && !a->ds))
    return MPFA_ERR_INVALID;
  size_t need = 0;
  if (mpfa_decode_workspace_size(a->batch, a->h_q, a->max_partitions, &need) != MPFA_OK)
    return MPFA_ERR_INVALID;

  p = mpfa::DecodeParams{};
  p.batch = a->batch;
  p.h_q = a->h_q;
  p.h_kv = a->h_kv;
  p.max_pages = a->max_pages;
  p.partition_tokens = a->partition_tokens;
  p.max_partitions = a->max_partitions;
  p.smooth = smooth;
  p.mx = (a->flags & MPFA_MXFP4) != 0;
  p.lam = kLambda;
  p.kv_len = a->kv_len;
  p.page_table = a->page_table;
  p.q_codes = a->q_codes;
  p.q_scales = a->q_scales;
  p.q_tscale = a->q_tscale;
  p.k_codes = a->k_codes;
  p.k_scales = a->k_scales;
  p.v_codes = a->v_codes;
  p.ds = static_cast<const uint16_t*>(a->ds);
  p.k_tscale = a->k_tscale;
  p.ws = nullptr;
  p.out = static_cast<uint16_t*>(a->out);
  return MPFA_OK;
}

// Decode arguments plus a caller-provided workspace of workspace_bytes.
static mpfa_status decode_params(const mpfa_decode_args* a, void* workspace, size_t workspace_bytes,
                                 mpfa::DecodeParams& p) {
  const mpfa_status st = decode_args_params(a, p);
  if (st != MPFA_OK) return st;
  size_t need = 0;
  mpfa_decode_workspace_size(a->batch, a->h_q, a->max_partitions, &need);
  if (!workspace || workspace_bytes < need) return MPFA_ERR_WORKSPACE;
  p.ws = static_cast<float*>(workspace);
  return MPFA_OK;
}


extern "C" {

const char* mpfa_status_string(mpfa_status s) {
  switch (s) {
    case MPFA_OK: return "ok";
    case MPFA_ERR_INVALID: return "invalid argument";
    case MPFA_ERR_UNSUPPORTED: return "unsupported configuration";
    case MPFA_ERR_WORKSPACE: return "workspace missing or too small";
    case MPFA_ERR_HIP: return "HIP runtime error";
    case MPFA_ERR_DATA: return "input data breaks a precondition (debug check)";
  }
  return "unknown status";
}

const char* mpfa_version(void) { return "mpfa-gfx950 0.1"; }

mpfa_status mpfa_quantize_qk(const mpfa_quant_args* a, mpfa_stream_t stream) {
  if (!a) return MPFA_ERR_INVALID;
  if (a->head_dim != MPFA_HEAD_DIM) return a->head_dim > 0 ? MPFA_ERR_UNSUPPORTED : MPFA_ERR_INVALID;
  if (a->batch < 1 || a->total_tokens < 0 || a->max_seqlen < 0 || a->num_pages < 1)
    return MPFA_ERR_INVALID;
  if (!heads_ok(a->h_q, a->h_kv)) return MPFA_ERR_INVALID;
  if (a->flags & ~(MPFA_SMOOTH | MPFA_COMPUTE_STATS | MPFA_TSCALE_UNIT | MPFA_MXFP4 | MPFA_PV_BF16 |
                   MPFA_PV_NVFP4))
    return MPFA_ERR_INVALID;
  const uint32_t pvq = a->flags & (MPFA_PV_BF16 | MPFA_PV_NVFP4);
  if (pvq == (MPFA_PV_BF16 | MPFA_PV_NVFP4) || (pvq && !a->v_aux)) return MPFA_ERR_INVALID;
  if (pvq && (a->flags & MPFA_MXFP4)) return MPFA_ERR_UNSUPPORTED;
  const bool smooth = a->flags & MPFA_SMOOTH;
  if (!a->cu_seqlens || !a->q || !a->k || !a->v || !a->slot_mapping || !a->q_mean || !a->k_mean ||
      !a->k_tscale || !a->q_codes || !a->q_scales || !a->q_tscale || !a->k_codes || !a->k_scales ||
      !a->v_codes || (smooth && !a->ds))
    return MPFA_ERR_INVALID;
  if ((int64_t)a->batch * (a->h_q + a->h_kv) > INT32_MAX) return MPFA_ERR_INVALID;
  if (a->batch > 65535) return MPFA_ERR_UNSUPPORTED;   // sequences run on the grid's y dimension

  mpfa::QuantParams p{};
  p.batch = a->batch;
  p.total_tokens = a->total_tokens;
  p.h_q = a->h_q;
  p.h_kv = a->h_kv;
  p.smooth = smooth;
  p.compute_stats = (a->flags & MPFA_COMPUTE_STATS) != 0;
  p.stats_k = p.compute_stats;
  p.tscale_unit = (a->flags & MPFA_TSCALE_UNIT) != 0;
  p.mx = (a->flags & MPFA_MXFP4) != 0;
  p.max_seqlen = a->max_seqlen;
  p.need_partials = (p.compute_stats && p.smooth) || !(p.tscale_unit || p.mx);
  p.cu_seqlens = a->cu_seqlens;
  p.q = static_cast<const uint16_t*>(a->q);
  p.k = static_cast<const uint16_t*>(a->k);
  p.v = static_cast<const uint16_t*>(a->v);
  p.slot_mapping = a->slot_mapping;
  p.q_mean = static_cast<uint16_t*>(a->q_mean);
  p.k_mean = static_cast<uint16_t*>(a->k_mean);
  p.k_tscale = a->k_tscale;
  p.q_codes = a->q_codes;
  p.q_scales = a->q_scales;
  p.q_tscale = a->q_tscale;
  p.k_codes = a->k_codes;
  p.k_scales = a->k_scales;
  p.v_codes = a->v_codes;
  p.ds = static_cast<uint16_t*>(a->ds);
  p.pv = (a->flags & MPFA_PV_BF16) ? 1 : (a->flags & MPFA_PV_NVFP4) ? 2 : 0;
  p.v_aux = static_cast<uint8_t*>(a->v_aux);
  p.num_pages = a->num_pages;
#ifdef MPFA_DEBUG_CHECKS
  const mpfa_status dst = check_quant(a, reinterpret_cast<hipStream_t>(stream));
  if (dst != MPFA_OK) return dst;
#endif
  return mpfa::launch_quantize(p, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? MPFA_OK
                                                                                        : MPFA_ERR_HIP;
}

mpfa_status mpfa_prefill(const mpfa_prefill_args* a, mpfa_stream_t stream) {
  mpfa::PrefillParams p;
  mpfa_status st = prefill_params(a, p);
  if (st != MPFA_OK) return st;
#ifdef MPFA_DEBUG_CHECKS
  st = check_prefill(a, reinterpret_cast<hipStream_t>(stream));
  if (st != MPFA_OK) return st;
#endif
  return mpfa::launch_prefill(p, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? MPFA_OK
                                                                                       : MPFA_ERR_HIP;
}

mpfa_status mpfa_decode_workspace_size(int32_t batch, int32_t h_q, int32_t max_partitions,
                                       size_t* bytes) {
  if (!bytes || batch < 1 || h_q < 1 || max_partitions < 1) return MPFA_ERR_INVALID;
  *bytes = (size_t)batch * (size_t)h_q * (size_t)max_partitions * (MPFA_HEAD_DIM + 2) * sizeof(float);
  return MPFA_OK;
}

mpfa_status mpfa_decode_choose_partition(int32_t batch, const int32_t* kv_len_host, int32_t h_kv,
                                         int32_t num_cus, int32_t* partition_tokens) {
  if (batch < 1 || !kv_len_host || h_kv < 1 || num_cus < 1 || !partition_tokens)
    return MPFA_ERR_INVALID;
  double total = 0.0;
  for (int b = 0; b < batch; ++b) {
    if (kv_len_host[b] < 1) return MPFA_ERR_INVALID;
    total += (double)kv_len_host[b] * h_kv;
  }
  // aim for about 32 partition waves per compute unit
  const double target_items = 32.0 * num_cus;
  int64_t part = (int64_t)std::ceil(total / target_items / 128.0) * 128;
  if (part < 256) part = 256;
  if (part > 16384) part = 16384;
  *partition_tokens = (int32_t)part;
  return MPFA_OK;
}

mpfa_status mpfa_decode_paged(const mpfa_decode_args* a, void* workspace, size_t workspace_bytes,
                              mpfa_stream_t stream) {
  mpfa::DecodeParams p;
  mpfa_status st = decode_params(a, workspace, workspace_bytes, p);
  if (st != MPFA_OK) return st;
#ifdef MPFA_DEBUG_CHECKS
  st = check_decode(a, reinterpret_cast<hipStream_t>(stream));
  if (st != MPFA_OK) return st;
#endif
  return mpfa::launch_decode(p, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? MPFA_OK
                                                                                      : MPFA_ERR_HIP;
}

mpfa_status mpfa_decode_paged_static(const mpfa_decode_args* a, mpfa_stream_t stream) {
  mpfa::DecodeParams p;
  mpfa_status st = decode_args_params(a, p);
  if (st != MPFA_OK) return st;
  size_t need = 0;
  mpfa_decode_workspace_size(a->batch, a->h_q, a->max_partitions, &need);
  if (need > MPFA_STATIC_SCRATCH_BYTES) return MPFA_ERR_WORKSPACE;
#ifdef MPFA_DEBUG_CHECKS
  st = check_decode(a, reinterpret_cast<hipStream_t>(stream));
  if (st != MPFA_OK) return st;
#endif
  void* ws = nullptr;
  if (mpfa::static_decode_scratch(&ws) != hipSuccess) return MPFA_ERR_HIP;
  p.ws = static_cast<float*>(ws);
  return mpfa::launch_decode(p, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? MPFA_OK
                                                                                      : MPFA_ERR_HIP;
}

mpfa_status mpfa_mixed_workspace_size(int32_t batch, int32_t h_q, int32_t h_kv, int32_t max_partitions,
                                      size_t* bytes) {
  size_t states = 0;
  if (!bytes || h_kv < 1 || mpfa_decode_workspace_size(batch, h_q, max_partitions, &states) != MPFA_OK)
    return MPFA_ERR_INVALID;
  *bytes = mixed_counter_offset(states) + (size_t)batch * (size_t)h_kv * sizeof(uint32_t);
  return MPFA_OK;
}

mpfa_status mpfa_mixed_step(const mpfa_prefill_args* prefill, const mpfa_decode_args* decode,
                            void* workspace, size_t workspace_bytes, mpfa_stream_t stream) {
  if (!prefill || !decode) return MPFA_ERR_INVALID;
  // the fused kernel runs the method's placements only (rank-one seed or none,
  // FP8 PV), with one smoothing / format setting for both parts
  if (prefill->flags & (MPFA_SEED_MFMA | MPFA_SEED_ELEMWISE | MPFA_PV_BF16 | MPFA_PV_NVFP4))
    return MPFA_ERR_UNSUPPORTED;
  if ((prefill->flags & (MPFA_SMOOTH | MPFA_MXFP4)) != (decode->flags & (MPFA_SMOOTH | MPFA_MXFP4)))
    return MPFA_ERR_INVALID;
  mpfa::MixedParams m{};
  mpfa_status st = prefill_params(prefill, m.pre);
  if (st != MPFA_OK) return st;
  size_t need = 0;
  if (mpfa_mixed_workspace_size(decode->batch, decode->h_q, decode->h_kv, decode->max_partitions, &need) !=
      MPFA_OK)
    return MPFA_ERR_INVALID;
  if (!workspace || workspace_bytes < need) return MPFA_ERR_WORKSPACE;
  st = decode_params(decode, workspace, workspace_bytes, m.dec);
  if (st != MPFA_OK) return st;
  size_t states = 0;
  mpfa_decode_workspace_size(decode->batch, decode->h_q, decode->max_partitions, &states);
  m.counters = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(workspace) + mixed_counter_offset(states));
  const int64_t n_pre = (int64_t)m.pre.n_qtiles * m.pre.h_q * m.pre.batch;
  const int64_t n_items = (int64_t)m.dec.batch * m.dec.h_kv * m.dec.max_partitions;
  const int64_t n_rounds = (n_items + 63) / 64;                  // decode rounds of 8 x 8 items
  const int64_t pre_rounds = (n_pre + 7) / 8;
  if (n_pre + 64 * n_rounds + 8 > INT32_MAX) return MPFA_ERR_INVALID;
  m.n_pre_blocks = (int)n_pre;
  m.n_dec_rounds = (int)n_rounds;
  // decode rounds first, back to back, then the prefill items (see mixed.hip)
  m.stride = 1;
  m.first = 0;
  m.n_blocks = (int)(8 * (pre_rounds + n_rounds));
#ifdef MPFA_DEBUG_CHECKS
  st = check_prefill(prefill, reinterpret_cast<hipStream_t>(stream));
  if (st == MPFA_OK) st = check_decode(decode, reinterpret_cast<hipStream_t>(stream));
  if (st != MPFA_OK) return st;
#endif
  return mpfa::launch_mixed(m, reinterpret_cast<hipStream_t>(stream)) == hipSuccess ? MPFA_OK
                                                                                    : MPFA_ERR_HIP;
}


mpfa_status mpfa_convert(int32_t fmt, const float* x, int64_t n, uint8_t* out, mpfa_stream_t stream) {
  const bool fmt_ok = (fmt >= 0 && fmt <= 3) || (fmt >= 0x101 && fmt <= 0x17E) || (fmt >= 0x201 && fmt <= 0x2FE) ||
                      (fmt >= 0x301 && fmt <= 0x37E) || (fmt >= 0x401 && fmt <= 0x4FE);
  if (!fmt_ok || n < 0 || (n > 0 && (!x || !out))) return MPFA_ERR_INVALID;
  if (n > (int64_t)UINT32_MAX * 256) return MPFA_ERR_INVALID;
  return mpfa::launch_convert(fmt, x, n, out, reinterpret_cast<hipStream_t>(stream)) == hipSuccess
             ? MPFA_OK
             : MPFA_ERR_HIP;
}

}  // extern "C"
