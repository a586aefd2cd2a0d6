// mpfa_internal.h -- launch parameter blocks shared by the host API layer and
// the gfx950 kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpfa {

constexpr int kMaxKvHeadsQuant = 32;
// decode batches up to this many sequences use the packed, XCD-rotated block
// map (each workgroup looks its work up with an O(batch) scan); larger ones a
// three-dimensional grid
constexpr int kDecodePackedMaxBatch = 512;
// size of the per-GPU device array that holds the decode partition states of
// mpfa_decode_paged_static (the entry point for callers that cannot allocate)
constexpr size_t kStaticScratchBytes = size_t(64) << 20;

struct QuantParams {
  int batch, total_tokens, max_seqlen, h_q, h_kv;
  int smooth, compute_stats, stats_k, tscale_unit;
  int need_partials;  // per-token statistics needed: means (STATS + SMOOTH) or amax (NVFP4 t)
  int mx;           // Q/K in MXFP4 (E8M0 per 32 channels, tensor scale 1)
  const int32_t* cu_seqlens;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int64_t* slot_mapping;
  uint16_t* q_mean;
  uint16_t* k_mean;
  float* k_tscale;
  uint8_t* q_codes;
  uint8_t* q_scales;
  float* q_tscale;
  uint8_t* k_codes;
  uint8_t* k_scales;
  uint8_t* v_codes;
  uint16_t* ds;
  int pv;           // 0: FP8 V only; 1: also BF16 V in v_aux; 2: also NVFP4 V in v_aux
  uint8_t* v_aux;
  int64_t num_pages;
};

struct PrefillParams {
  int batch, h_q, h_kv, max_pages;
  int n_qtiles;     // max query tiles of one sequence
  int smooth;
  int seed_mfma;    // 1: compensation formed by the rank-one BF16 MFMA, 0: accumulator input
  int seed_elem;    // 1: compensation added to each score after the QK product
  int mx;           // Q/K in MXFP4: QK on the scaled FP4 MFMA
  int xcd_remap;    // 1: spread KV heads over the 8 XCDs (needs h_kv % 8 == 0)
  float lam;        // log2(e) / sqrt(128)
  const int32_t* cu_seqlens_q;
  const int32_t* q_start;
  const int32_t* kv_len;
  const int32_t* page_table;
  const uint8_t* q_codes;
  const uint8_t* q_scales;
  const float* q_tscale;
  const uint8_t* k_codes;
  const uint8_t* k_scales;
  const uint8_t* v_codes;
  const uint16_t* ds;
  const float* k_tscale;
  uint16_t* out;
  int pv;           // 0: FP8 P and V; 1: BF16 P and V (v_aux); 2: NVFP4 P and V (v_aux)
  const uint8_t* v_aux;
  int64_t num_pages;
};

struct DecodeParams {
  int batch, h_q, h_kv, max_pages;
  int partition_tokens, max_partitions;
  int smooth;
  int mx;           // Q/K in MXFP4: QK on the scaled FP4 MFMA
  float lam;
  const int32_t* kv_len;
  const int32_t* page_table;
  const uint8_t* q_codes;
  const uint8_t* q_scales;
  const float* q_tscale;
  const uint8_t* k_codes;
  const uint8_t* k_scales;
  const uint8_t* v_codes;
  const uint16_t* ds;
  const float* k_tscale;
  float* ws;        // [batch][h_q][max_partitions][130]: m*lambda', l, O[128]
  uint16_t* out;
};

// One launch for a step of prefill items and decode partitions (with the merge).
struct MixedParams {
  PrefillParams pre;
  DecodeParams dec;
  int n_pre_blocks;   // prefill work items (query tiles x heads x sequences)
  int n_dec_rounds;   // rounds of 8 decode groups (a group is 8 decode work items)
  int first;          // round index of the first decode round
  int stride;         // rounds of 8 blocks from one decode round to the next
  int n_blocks;       // grid size
  uint32_t* counters; // [dec.batch][dec.h_kv] partition counters, zero between calls
};

hipError_t launch_quantize(const QuantParams& p, hipStream_t stream);
hipError_t launch_scan_nonfinite(const uint16_t* x, int64_t n, int* flag, hipStream_t stream);
hipError_t launch_mixed(const MixedParams& m, hipStream_t stream);
hipError_t launch_convert(int fmt, const float* x, int64_t n, uint8_t* out, hipStream_t stream);
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream);
hipError_t launch_decode(const DecodeParams& p, hipStream_t stream);
// Device address of the static decode scratch array on the current device
// (looked up once per device, then cached).
hipError_t static_decode_scratch(void** ptr);

}  // namespace mpfa
