/*
 * mpfa.h -- C ABI of the MI355X (gfx950) QK4PV8 FlashAttention library.
 *
 * The method (MpFA, "QK4PV8"): Q and K are centered per sequence and head and
 * quantized to NVFP4 (E2M1 elements, one E4M3 scale per 16 head-dimension
 * elements, Sec. 2.1 Eq. 1 and Sec. 4.1-4.2); the removed Q-mean term is
 * restored as a rank-one contraction that seeds the score accumulator
 * (Sec. 4.3 Eqs. 8-11); online softmax runs in FP32 (Sec. 2.2 Eqs. 3-6); P is
 * quantized to FP8 E4M3 with the fixed scale 448 (Sec. 4.1); V is stored in
 * FP8 E4M3 and PV runs on FP8 matrix cores; KV blocks are visited in reverse
 * (Sec. 4.1).  Prefill is causal (Algorithm 1); decode is split-KV over a
 * paged cache with a log-sum-exp merge (Sec. 5.3, Sec. 6).
 *
 * Conventions for every entry point:
 *  - Argument structs are host memory.  Every pointer inside them is DEVICE
 *    memory owned by the caller; the library keeps no reference after return.
 *  - bf16 tensors are passed as raw 16-bit patterns (void*).
 *  - All shape and flag validation happens on the host before any HIP call;
 *    a rejected call launches nothing and returns MPFA_ERR_INVALID (bad
 *    value, null pointer) or MPFA_ERR_UNSUPPORTED (valid but not built, e.g.
 *    head_dim != 128).  Launch failures return MPFA_ERR_HIP.
 *  - Work is enqueued asynchronously on `stream` (0 = default stream); no
 *    host synchronisation and no device allocation happen inside
 *    mpfa_prefill and mpfa_decode_paged, so both may be captured in a HIP
 *    graph.  mpfa_quantize_qk does not allocate either.
 *  - Data-dependent conditions (page index out of range, non-finite inputs,
 *    kv_len larger than the page table) are NOT checked by the release
 *    library (libmpfa.so): the caller guarantees them.  The debug library
 *    (libmpfa_debug.so, same ABI) checks them before launching anything and
 *    returns MPFA_ERR_DATA: it copies cu_seqlens, q_start, kv_len, the page
 *    table rows in use and slot_mapping to the host, scans Q/K/V for
 *    non-finite values on the device, and so synchronizes the stream and
 *    allocates a 4-byte flag per call.  Checked: sequence lengths consistent
 *    with cu_seqlens / total_tokens / max_seqlen; slots in [0, 64 num_pages);
 *    q_start >= 0 and q_start + query tokens <= kv_len <= 64 max_pages; decode
 *    kv_len >= 1 and within max_partitions partitions; page-table entries of
 *    the pages in use >= 0, and < num_pages when the arguments carry it.
 *  - The library holds no mutable global state apart from the per-GPU scratch
 *    of mpfa_decode_paged_static; concurrent calls of the other entry points
 *    on different streams are safe when their output buffers do not overlap.
 *
 * Layouts (head_dim D = 128, 16-element NVFP4 groups, 64-token pages):
 *  - Q, K, V inputs: bf16 [T][H][128], tokens of all sequences packed,
 *    sequence b owning tokens cu_seqlens[b] .. cu_seqlens[b+1]-1.
 *  - NVFP4 rows: 64 code bytes (channel 2i in the low nibble of byte i,
 *    channel 2i+1 in the high nibble) + 8 E4M3 scale bytes (group g covers
 *    channels 16g .. 16g+15) + one FP32 power-of-two tensor scale per
 *    (sequence, head).  Value of channel c: t * e4m3(scale[c/16]) * e2m1(code).
 *  - Paged cache, page p, KV head h, token slot o (0..63):
 *      k_codes  u8   [P][H_kv][64][64]
 *      k_scales u8   [P][H_kv][64][8]
 *      v_codes  u8   [P][H_kv][128][64]   (channel-major: [channel][slot])
 *      ds       bf16 [P][H_q][64]         (Delta_S side cache, smoothing only)
 *    A token's slot is slot_mapping = page * 64 + o.
 *  - page_table i32 [batch][max_pages]: logical page i of sequence b is
 *    physical page page_table[b * max_pages + i]; key position j of the
 *    sequence lives in logical page j / 64, slot j % 64.
 *  - Query head h uses KV head h / (H_q / H_kv).
 */
#ifndef MPFA_H
#define MPFA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* mpfa_stream_t;   /* == hipStream_t */

typedef enum {
    MPFA_OK = 0,
    MPFA_ERR_INVALID = 1,      /* bad argument value or null pointer          */
    MPFA_ERR_UNSUPPORTED = 2,  /* valid request this build does not implement */
    MPFA_ERR_WORKSPACE = 3,    /* workspace missing or too small              */
    MPFA_ERR_HIP = 4,          /* a HIP launch or runtime call failed         */
    MPFA_ERR_DATA = 5          /* debug build only: the contents of an input
                                  break a precondition (see below)            */
} mpfa_status;

#define MPFA_HEAD_DIM 128
#define MPFA_PAGE_TOKENS 64
#define MPFA_KV_TILE 128
#define MPFA_MAX_HEADS 256

/* flags */
#define MPFA_SMOOTH        1u  /* sequence centering + Delta_S compensation (off = "direct");
                                  prefill starts each QK accumulator at the rank-one term
                                  1 Delta_S^T (Sec. 4.3 Eq. 11) loaded as the MFMA
                                  accumulator input                                         */
#define MPFA_COMPUTE_STATS 2u  /* compute means and K tensor scales from this call's tokens  */
#define MPFA_TSCALE_UNIT   4u  /* NVFP4 tensor scale fixed to 1 (Eq. 1 without a 2nd level) */
#define MPFA_SEED_MFMA     8u  /* prefill: form the rank-one term 1 Delta_S^T with one BF16
                                  MFMA per 16-key block (Delta_S in reduction slot 0, ones
                                  in B), the paper's formulation (Sec. 5.2), instead of
                                  loading it as the accumulator input; bit-identical       */
#define MPFA_SEED_ELEMWISE 32u /* prefill: the placement the rank-one seed replaces (Sec. 3.2,
                                  Sec. 7.4 Fig. 10), kept for comparison: the QK accumulator
                                  starts at zero and Delta_S is added to every score in FP32
                                  after the product, before masking.  Agrees with the seeded
                                  placements up to FP32 rounding order (not bit-identical).
                                  Exclusive with MPFA_SEED_MFMA.                          */
#define MPFA_PV_BF16      64u  /* quantize + prefill: precision assignment NVFP4(QK) + BF16(PV)
                                  of the characterization in Sec. 3.1 / Fig. 3a: the
                                  quantizer also stores V in BF16 in v_aux (bf16
                                  [P][H_kv][128][64], channel-major like v_codes), and the
                                  prefill rounds P to BF16 (no scale) and runs PV on the
                                  BF16 MFMA over v_aux.  Not with MPFA_MXFP4,
                                  MPFA_SEED_MFMA or MPFA_SEED_ELEMWISE; decode: unsupported. */
#define MPFA_PV_NVFP4    128u  /* quantize + prefill: NVFP4(QK) + NVFP4(PV), the other arm of
                                  Fig. 3a: the quantizer stores V as NVFP4 in 16-key groups
                                  per channel in v_aux (a code plane u8 [P][H_kv][128][32],
                                  key 2i in the low nibble of byte i, then a scale plane u8
                                  [P][H_kv][128][4] of E4M3 group scales, tensor scale 1);
                                  the prefill quantizes P' = 2688 P per 16 keys with dynamic
                                  E4M3 scales (amax / 6) and runs PV on FP16 MFMA over the
                                  exactly dequantized operands.  Quantizer precondition: the
                                  call is a fresh prefill (token i of a sequence at slot
                                  i % 64 of its i / 64-th page); each page it touches is
                                  written whole, absent slots as zero.  Same exclusions as
                                  MPFA_PV_BF16.                                             */
#define MPFA_MXFP4        16u  /* Q/K in MXFP4 instead of NVFP4 (quantize, prefill, decode):
                                  one E8M0 scale per 32 channels (scale bytes 0..3 of the
                                  8-byte scale row; bytes 4..7 zero), tensor scales 1, and
                                  QK on the scaled FP4 MFMA.  All calls on one cache must
                                  agree on this flag.                                      */

/* ------------------------------------------------------------------------ */
/* Quantization / cache-write pass (Algorithm 1 stage one; Sec. 4.2, 4.3, 6) */
/* ------------------------------------------------------------------------ */
/*
 * For each sequence b of the call:
 *  - with MPFA_COMPUTE_STATS: Qbar, Kbar = per-(head, channel) means over the
 *    call's tokens (Eq. 7), summed in FP32 sequentially inside 128-token
 *    blocks and then over the block partials in order, divided in FP32 and
 *    rounded to BF16 (written to q_mean / k_mean; zero without MPFA_SMOOTH);
 *    k_tscale[b][h] = smallest 2^k (k in [-63, 63]) with 2688 * 2^k >= max
 *    |K - Kbar| over the call's tokens (1 if that max is 0 or with
 *    MPFA_TSCALE_UNIT).  Without the flag the means and k_tscale are read
 *    (frozen after the first prefill, Sec. 6).
 *  - q_tscale[b][h]: the same rule over this call's centered Q tokens.
 *  - Q_c = Q - Qbar and K_c = K - Kbar in FP32; NVFP4 per 16-channel group:
 *    scale = E4M3_RNE_sat(amax / (6 t)), codes = E2M1_RNE_sat(x / (t * scale))
 *    with IEEE FP32 divisions; a group whose scale is 0 stores sign-only codes.
 *  - With MPFA_MXFP4 (the 32-element E8M0 block format Sec. 2.1 names next to
 *    NVFP4): tensor scales are 1; per 32-channel block X = 2^e with
 *    e = floor(log2 amax) - 2 clamped to [-127, 127] (e = -127 for an all-zero
 *    block), scale byte e + 127, codes = E2M1_RNE_sat(x / X).
 *  - V is stored as E4M3_RNE_sat(V) (no scale, not centered, Sec. 4.2).
 *  - With MPFA_SMOOTH, ds[slot][h_q] = BF16_RNE(sum_c Qbar[h_q][c] * K_c[c])
 *    as an FP32 fused multiply-add chain over c = 0..127 (Eq. 9).
 * Writes q_codes/q_scales rows of this call's tokens and the cache slots given
 * by slot_mapping.  Deterministic: identical inputs give identical bytes.
 */
typedef struct {
    int32_t batch;            /* sequences in this call, 1 .. 65535                */
    int32_t total_tokens;     /* T = cu_seqlens[batch] (host copy)               */
    int32_t max_seqlen;       /* host: max tokens of one sequence in this call   */
    int32_t h_q, h_kv;        /* heads; h_q % h_kv == 0, h_q <= MPFA_MAX_HEADS   */
    int32_t head_dim;         /* must be 128                                     */
    uint32_t flags;           /* MPFA_SMOOTH | MPFA_COMPUTE_STATS | MPFA_TSCALE_UNIT | MPFA_MXFP4
                                 | MPFA_PV_BF16 or MPFA_PV_NVFP4 */
    int64_t num_pages;        /* cache capacity in pages (slot_mapping < 64 * num_pages) */
    const int32_t* cu_seqlens;   /* [batch+1]                                    */
    const void* q;               /* bf16 [T][h_q][128]                           */
    const void* k;               /* bf16 [T][h_kv][128]                          */
    const void* v;               /* bf16 [T][h_kv][128]                          */
    const int64_t* slot_mapping; /* [T]                                          */
    void* q_mean;                /* bf16 [batch][h_q][128]   (out with STATS, else in) */
    void* k_mean;                /* bf16 [batch][h_kv][128]  (out with STATS, else in) */
    float* k_tscale;             /* [batch][h_kv]            (out with STATS, else in) */
    uint8_t* q_codes;            /* out [T][h_q][64]                             */
    uint8_t* q_scales;           /* out [T][h_q][8]                              */
    float* q_tscale;             /* out [batch][h_q]                             */
    uint8_t* k_codes;            /* cache, see layouts                           */
    uint8_t* k_scales;
    uint8_t* v_codes;
    void* ds;                    /* bf16 cache; may be NULL without MPFA_SMOOTH  */
    void* v_aux;                 /* with MPFA_PV_BF16 / MPFA_PV_NVFP4 (see there); else
                                    ignored (may be NULL)                          */
} mpfa_quant_args;

mpfa_status mpfa_quantize_qk(const mpfa_quant_args* args, mpfa_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Causal prefill (Algorithm 1 main loop; Sec. 5.1, 5.2)                      */
/* ------------------------------------------------------------------------ */
/*
 * Query i of sequence b (token cu_seqlens[b] + i, absolute position
 * q_start[b] + i) attends to keys 0 .. q_start[b] + i of the sequence's paged
 * cache.  KV tiles of 128 keys (multiples of 128) are visited from the
 * query's own tile down to tile 0.  For every tile:
 *   S = 1 * Delta_S (rank-one seed, with MPFA_SMOOTH)
 *       + dequant(Q_hat) dequant(K_hat)^T,  masked after the seed;
 *   m' = max(m, rowmax S); P = 2^(lambda (S - m')), lambda = log2(e)/sqrt(128);
 *   l = 2^(lambda (m - m')) l + rowsum P;  P_hat = E4M3(448 P);
 *   O = 2^(lambda (m - m')) O + P_hat V_hat.
 * Output out[token][h][:] = BF16(O / (448 l)).  Requires
 * q_start[b] + (cu_seqlens[b+1] - cu_seqlens[b]) <= kv_len[b].
 * The NVFP4 products are computed exactly (FP16 operands hold t-free
 * scale * element values exactly); accumulation is FP32.
 */
typedef struct {
    int32_t batch, h_q, h_kv, head_dim;
    int32_t max_seqlen_q;     /* host: max query tokens of one sequence          */
    int32_t max_pages;        /* page_table row length                           */
    uint32_t flags;           /* MPFA_SMOOTH, MPFA_SEED_MFMA or MPFA_SEED_ELEMWISE, MPFA_MXFP4,
                                 MPFA_PV_BF16 or MPFA_PV_NVFP4                   */
    const int32_t* cu_seqlens_q; /* [batch+1] query tokens                       */
    const int32_t* q_start;   /* [batch] absolute position of query 0            */
    const int32_t* kv_len;    /* [batch] keys in the cache (>= q_start + n_q)    */
    const int32_t* page_table;/* [batch][max_pages]                              */
    const uint8_t* q_codes;   /* [T][h_q][64]                                    */
    const uint8_t* q_scales;  /* [T][h_q][8]                                     */
    const float* q_tscale;    /* [batch][h_q]                                    */
    const uint8_t* k_codes;
    const uint8_t* k_scales;
    const uint8_t* v_codes;
    const void* ds;           /* bf16 side cache (MPFA_SMOOTH)                   */
    const float* k_tscale;    /* [batch][h_kv]                                   */
    void* out;                /* bf16 [T][h_q][128]                              */
    const void* v_aux;        /* with MPFA_PV_BF16 / MPFA_PV_NVFP4; else ignored */
    int64_t num_pages;        /* cache capacity in pages (plane offset of an NVFP4
                                 v_aux); read with MPFA_PV_NVFP4 and by the debug
                                 library's page index check (0 = not given)       */
} mpfa_prefill_args;

mpfa_status mpfa_prefill(const mpfa_prefill_args* args, mpfa_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Split-KV paged decode (Sec. 5.3, Sec. 6)                                   */
/* ------------------------------------------------------------------------ */
/*
 * One query token per sequence (q rows indexed by sequence b), attending to
 * all kv_len[b] keys (the new token included; it must already be in the
 * cache).  Keys are split into partitions of partition_tokens keys
 * ([p*P, (p+1)*P)); each partition is visited in 128-key tiles from last to
 * first with its own (m, l, O), exactly as in prefill, and the partition
 * states are merged by log-sum-exp:
 *   M = max_p m_p; l = sum_p 2^(lambda (m_p - M)) l_p;
 *   O = sum_p 2^(lambda (m_p - M)) O_p; out = BF16(O / (448 l)).
 * The G = H_q / H_kv query heads of one KV head share one pass over the KV
 * partition (GQA packing); the compensation becomes a rank-G seed.
 * workspace: caller-owned device memory of at least
 * mpfa_decode_workspace_size(...) bytes; its contents on entry are ignored.
 * Launch limit: for batch <= 512, batch * ceil(max_partitions / 4) * (h_kv
 * rounded up to 8) workgroups of 256 threads must stay below 2^32 threads,
 * else MPFA_ERR_UNSUPPORTED (larger batches use a three-dimensional grid).
 */
typedef struct {
    int32_t batch, h_q, h_kv, head_dim;
    int32_t max_pages;
    int32_t partition_tokens; /* multiple of 128                                  */
    int32_t max_partitions;   /* >= ceil(max_b kv_len[b] / partition_tokens)      */
    uint32_t flags;           /* MPFA_SMOOTH, MPFA_MXFP4                          */
    const int32_t* kv_len;    /* [batch], each >= 1                               */
    const int32_t* page_table;/* [batch][max_pages]                               */
    const uint8_t* q_codes;   /* [batch][h_q][64]                                 */
    const uint8_t* q_scales;  /* [batch][h_q][8]                                  */
    const float* q_tscale;    /* [batch][h_q]                                     */
    const uint8_t* k_codes;
    const uint8_t* k_scales;
    const uint8_t* v_codes;
    const void* ds;
    const float* k_tscale;    /* [batch][h_kv]                                    */
    void* out;                /* bf16 [batch][h_q][128]                           */
    int64_t num_pages;        /* cache capacity in pages, 0 = not given; only the
                                 debug library reads it (page index check)        */
} mpfa_decode_args;

/* Bytes of decode workspace: batch * h_q * max_partitions * (128 + 2) * 4. */
mpfa_status mpfa_decode_workspace_size(int32_t batch, int32_t h_q, int32_t max_partitions,
                                       size_t* bytes);

/* Host helper: choose partition_tokens (a multiple of 128) for a batch so
 * that the number of (sequence, KV head, partition) work items is a few
 * times the compute-unit count; kv_len_host is host memory [batch]. */
mpfa_status mpfa_decode_choose_partition(int32_t batch, const int32_t* kv_len_host, int32_t h_kv,
                                         int32_t num_cus, int32_t* partition_tokens);

mpfa_status mpfa_decode_paged(const mpfa_decode_args* args, void* workspace, size_t workspace_bytes,
                              mpfa_stream_t stream);

/* Size of the library's own decode scratch on each GPU (partition states of
 * mpfa_decode_paged_static). */
#define MPFA_STATIC_SCRATCH_BYTES (64u << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * mpfa_decode_paged without the workspace argument.  The same kernels keep
 * their partition states in a device array of MPFA_STATIC_SCRATCH_BYTES that
 * the library holds on each GPU it runs on until the process ends; the caller
 * still passes the inputs and the output.  The call allocates nothing: its
 * first call on a device only looks up that device's address of the array.
 * Arguments, layouts and results are exactly those of mpfa_decode_paged.
 * Errors: as mpfa_decode_paged, and MPFA_ERR_WORKSPACE, before any launch,
 * when mpfa_decode_workspace_size(batch, h_q, max_partitions) exceeds
 * MPFA_STATIC_SCRATCH_BYTES.  Every call on a GPU shares that GPU's array:
 * calls that overlap on one GPU (concurrent streams, or threads) race and
 * must be serialized by the caller; the array keeps the last call's states,
 * and no call needs it to start at any particular value.
 */
mpfa_status mpfa_decode_paged_static(const mpfa_decode_args* args, mpfa_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Mixed serving step in one launch (Sec. 7.3; prefill and decode requests    */
/* of one step served together)                                               */
/* ------------------------------------------------------------------------ */
/*
 * Runs the causal prefill described by `prefill` and the split-KV decode
 * described by `decode` in a single kernel launch, merge included (the last
 * partition of each (sequence, KV head) merges its query heads): decode
 * partitions first, then the prefill query tiles, in one grid.
 * Results are bit-identical to mpfa_prefill followed by mpfa_decode_paged
 * with the same arguments.  Both parts must use the same MPFA_SMOOTH /
 * MPFA_MXFP4 setting (else MPFA_ERR_INVALID); the prefill flags may not
 * contain MPFA_SEED_MFMA, MPFA_SEED_ELEMWISE or the PV characterization
 * flags (MPFA_ERR_UNSUPPORTED).  Each part is validated as by its own entry
 * point.
 * workspace: caller-owned device memory of at least
 * mpfa_mixed_workspace_size(decode batch, h_q, h_kv, max_partitions) bytes:
 * the decode partition states, then one 32-bit counter per (sequence, KV
 * head).  The counters must be zero before the first call on a workspace
 * (allocate it zeroed); every completed call leaves them zero again.  Calls
 * that share a workspace must not overlap.
 */
mpfa_status mpfa_mixed_workspace_size(int32_t batch, int32_t h_q, int32_t h_kv,
                                      int32_t max_partitions, size_t* bytes);
mpfa_status mpfa_mixed_step(const mpfa_prefill_args* prefill, const mpfa_decode_args* decode,
                            void* workspace, size_t workspace_bytes, mpfa_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Utilities                                                                  */
/* ------------------------------------------------------------------------ */
/* Element-wise device conversions, exposed so that their rounding can be
 * checked exhaustively: fmt 0 = FP32 -> E4M3 (RNE, saturating at 448, sign
 * kept), fmt 1 = FP32 -> E2M1 (RNE, saturating at 6, sign kept, one code per
 * output byte), both written out from the format definitions; fmt 2 and 3 =
 * the same two conversions through the gfx950 hardware converters, as the
 * quantization pass uses them (must give identical bytes); 0x100 + c (c =
 * 1..126, a positive E4M3 code) = the E2M1 code of x / e4m3(c) exactly as the
 * NVFP4 quantizer forms it (the correctly rounded quotient, then E2M1);
 * 0x200 + b (b = 1..254) = the E2M1 code of x / 2^(b - 127) as the MXFP4
 * quantizer forms it; 0x300 + c and 0x400 + b = the same two quotients
 * written out from their definitions (IEEE division __fdiv_rn, exact
 * power-of-two scaling ldexpf, then the fmt 1 encoder), the references the
 * quantizer's element paths are checked against.  x and out are device
 * pointers of n elements; x must be finite (the codes of NaN inputs are
 * unspecified, as everywhere in the library); MPFA_ERR_INVALID for another
 * fmt. */
mpfa_status mpfa_convert(int32_t fmt, const float* x, int64_t n, uint8_t* out,
                         mpfa_stream_t stream);

const char* mpfa_status_string(mpfa_status status);

/* Library version string (static storage). */
const char* mpfa_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MPFA_H */
