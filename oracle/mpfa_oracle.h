/*
 * mpfa_oracle.h -- plain, slow CPU oracle for QK4PV8 FlashAttention (MpFA).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product path
 * (the HIP library behind include/mpfa.h) never calls it, and the two share
 * no code, headers, tables or helpers.
 *
 * Everything between the method's rounding points is evaluated in FP64.
 * The rounding points are:
 *   R2  per-(sequence, head) means rounded to BF16            (Sec. 4.2, Eq. 7)
 *   R3  NVFP4 block scale rounded to E4M3                     (Sec. 2.1, Eq. 1)
 *   R4  NVFP4 elements rounded to E2M1                        (Sec. 2.1, Eq. 1)
 *   R5  V rounded to FP8 E4M3                                 (Sec. 4.1, Sec. 4.2)
 *   R6  compensation vector Delta_S rounded to BF16           (Sec. 4.3, Eqs. 9 and 11)
 *   R7  P rounded to FP8 E4M3 with the fixed scale 448        (Sec. 4.1)
 *   R8  output rounded to BF16                                (Algorithm 1, output)
 *
 * Layouts follow the C-ABI of the product library (head_dim 128, 16-element
 * NVFP4 groups, 64-token cache pages, 128-key tiles) so that codes can be
 * compared byte for byte; the oracle re-derives them from the paper's
 * definitions, not from the product code.
 *
 * Functions without a dedicated pin are marked "parity unpinned" in their
 * comment; the full quantized output values are such a case (the paper
 * prints no worked numeric example).
 */
#ifndef MPFA_ORACLE_H
#define MPFA_ORACLE_H

#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_D      128   /* head dimension                        */
#define ORC_G      16    /* NVFP4 group along the head dimension  */
#define ORC_NG     8     /* groups per head row                   */
#define ORC_PAGE   64    /* tokens per cache page                 */

/* ---- mode flags ---------------------------------------------------------- */
#define ORC_SMOOTH        1   /* sequence centering + Delta_S compensation   */
#define ORC_COMPUTE_STATS 2   /* compute means / tensor scales (first prefill) */
#define ORC_TSCALE_UNIT   4   /* tensor scale fixed to 1 (Eq. 1 literally)   */
#define ORC_MXFP4         8   /* Q/K as MXFP4: E8M0 scale per 32, tensor scale 1
                                 (also set in orc_cache.flags for the attention) */

#define ORC_PV_BF16      16   /* characterization of Sec. 3.1 / Fig. 3a: V kept in BF16
                                 (cache array v_aux) and P rounded to BF16          */
#define ORC_PV_NVFP4     32   /* characterization of Sec. 3.1 / Fig. 3a: V as NVFP4 in
                                 16-key groups per channel (v_aux, tensor scale 1) and
                                 P as NVFP4 with dynamic E4M3 scales per 16 keys     */
#define ORC_QUANT_P       1   /* attention core: round 448*P to E4M3         */
#define ORC_REVERSE       2   /* attention core: visit KV tiles last to first */
#define ORC_P_BF16        4   /* attention core: round P to BF16 (no scale)  */
#define ORC_P_NVFP4       8   /* attention core: 2688*P as NVFP4 per 16 keys aligned to
                                 multiples of 16: E4M3 scale of amax/6, E2M1 codes  */

/* ---- number formats (Sec. 2.1 Eq. 1, Sec. 4.1) ----------------------------- */
double  orc_e2m1_value(uint8_t code);            /* code in 0..15, bit 3 = sign */
uint8_t orc_e2m1_encode(double y);               /* RNE on the E2M1 grid, saturating at 6 */
double  orc_e4m3_value(uint8_t code);            /* OCP E4M3 (FN): max 448, 0x7F/0xFF NaN */
uint8_t orc_e4m3_encode(double x);               /* RNE, saturating at 448 */
float   orc_bf16_value(uint16_t bits);
uint16_t orc_bf16_encode(float x);               /* RNE (finite inputs) */
uint16_t orc_bf16_encode_f64(double x);          /* RNE, one rounding from FP64 */

/* array helpers (used by exhaustive sweeps) */
void orc_e4m3_encode_f32_array(const float* x, int64_t n, uint8_t* out);
void orc_e2m1_encode_f32_array(const float* x, int64_t n, uint8_t* out);
void orc_bf16_encode_f32_array(const float* x, int64_t n, uint16_t* out);

/* ---- quantization pass (Algorithm 1 stage one; Sec. 4.2, 4.3, 6) ----------- */

/* Statistics for one (sequence, head): FP32 two-level sum, FP32 divide, BF16.
 * x: bf16 [n_tok] rows with row stride `stride` elements, 128 channels each.
 * mean_out: bf16[128].  When smooth == 0 the mean is zero.
 * tscale_out: power-of-two tensor scale (see orc_tensor_scale).            */
void orc_stats_one(const uint16_t* x, int64_t n_tok, int64_t stride, int smooth,
                   int tscale_unit, uint16_t* mean_out, float* tscale_out);

/* Smallest power of two t = 2^k (k clamped to [-63, 63], so that tQ * tK and
 * its inverse are normal FP32 numbers) with 2688 * t >= amax; 1 when amax == 0. */
float orc_tensor_scale(float amax);

/* NVFP4 quantization of one 128-channel row of centered FP32 values:
 * 8 E4M3 group scales and 64 bytes of packed E2M1 codes (even channel in the
 * low nibble). */
void orc_nvfp4_row(const float* xc, float t, uint8_t* codes64, uint8_t* scales8);

typedef struct {
    int32_t  batch, total_tokens, h_q, h_kv;
    int32_t  flags;                 /* ORC_SMOOTH | ORC_COMPUTE_STATS | ORC_TSCALE_UNIT */
    const int32_t*  cu_seqlens;     /* [batch+1] tokens of this call           */
    const uint16_t* q;              /* bf16 [T][h_q][128]                      */
    const uint16_t* k;              /* bf16 [T][h_kv][128]                     */
    const uint16_t* v;              /* bf16 [T][h_kv][128]                     */
    const int64_t*  slot_mapping;   /* [T] page*64 + offset                    */
    /* statistics: written when ORC_COMPUTE_STATS, else read (frozen)          */
    uint16_t* q_mean;               /* bf16 [batch][h_q][128]                  */
    uint16_t* k_mean;               /* bf16 [batch][h_kv][128]                 */
    float*    k_tscale;             /* [batch][h_kv]                           */
    /* outputs                                                                 */
    uint8_t* q_codes;               /* [T][h_q][64]                            */
    uint8_t* q_scales;              /* [T][h_q][8]                             */
    float*   q_tscale;              /* [batch][h_q]                            */
    uint8_t* k_codes;               /* [pages][h_kv][64][64]                   */
    uint8_t* k_scales;              /* [pages][h_kv][64][8]                    */
    uint8_t* v_codes;               /* [pages][h_kv][128][64]  channel-major   */
    uint16_t* ds;                   /* bf16 [pages][h_q][64]; unused w/o smooth */
    void*     v_aux;                /* ORC_PV_BF16: bf16 [pages][h_kv][128][64];
                                       ORC_PV_NVFP4: a code plane u8 [pages][h_kv][128][32]
                                       (key 2i in the low nibble of byte i) followed by
                                       a scale plane u8 [pages][h_kv][128][4] (E4M3 of
                                       keys 16j..16j+15).  NVFP4 needs
                                       each sequence's tokens at slots 0, 1, 2, ... of
                                       its pages in order (a fresh prefill); the call's
                                       pages are written whole, absent slots as zero.  */
    int64_t   num_pages;            /* cache capacity in pages (plane size of v_aux)    */
} orc_quant_args;

int orc_quantize_qk(const orc_quant_args* a);

/* ---- attention core (Algorithm 1 main loop, Sec. 2.2 Eqs. 3-6, Sec. 4.1) --- */

/* Online-softmax state of one query row. */
typedef struct { double m, l; double o[ORC_D]; } orc_state;

void orc_state_init(orc_state* s);

/* Visit keys [key_lo, key_hi) in tiles of `tile` keys aligned to multiples of
 * `tile` (absolute key index), last to first when ORC_REVERSE is set.
 * qd: FP64 query row; kd/vd: FP64 rows [key][128] indexed by absolute key;
 * dsd: FP64 compensation per key (NULL = none); keys > q_pos are masked.
 * O accumulates dec(P_hat) * v when ORC_QUANT_P (units of 1/448), else P * v. */
void orc_visit(orc_state* st, const double* qd, const double* kd, const double* vd,
               const double* dsd, int64_t q_pos, int64_t key_lo, int64_t key_hi,
               int tile, int flags);

/* Log-sum-exp merge of partition states, then divide by p_scale * l, where
 * p_scale is the factor the P quantizer applied (448, 2688 or 1) (Sec. 5.3). */
void orc_merge(const orc_state* parts, int n, double* out /*[128]*/, double p_scale);

/* Generic FP64 attention over contiguous arrays (used by the pins):
 * q [nq][128], k/v [nk][128], ds [nq][nk] or NULL, q_pos[nq] (keys > q_pos
 * masked; use nk-1 for no mask).  Each row is split into partitions of
 * `partition` keys (0 = one partition), each visited in `tile`-key tiles.
 * out [nq][128] FP64 (before the BF16 rounding R8). */
void orc_attention_f64(const double* q, const double* k, const double* v,
                       const double* ds, const int64_t* q_pos, int64_t nq, int64_t nk,
                       int tile, int64_t partition, int flags, double* out);

/* Textbook two-pass softmax attention in FP64 (Sec. 2.2 Eq. 2), scale 1/sqrt(d). */
void orc_attention_textbook(const double* q, const double* k, const double* v,
                            const int64_t* q_pos, int64_t nq, int64_t nk, double* out);

/* ---- product-shaped attention over the quantized paged cache -------------- */
typedef struct {
    int32_t batch, h_q, h_kv, max_pages, flags;  /* ORC_SMOOTH, ORC_MXFP4, ORC_PV_* */
    const int32_t*  page_table;   /* [batch][max_pages]                    */
    const int32_t*  kv_len;       /* [batch]                               */
    const uint8_t*  k_codes;      /* [pages][h_kv][64][64]                 */
    const uint8_t*  k_scales;     /* [pages][h_kv][64][8]                  */
    const uint8_t*  v_codes;      /* [pages][h_kv][128][64]                */
    const uint16_t* ds;           /* [pages][h_q][64] bf16 (smooth only)   */
    const float*    k_tscale;     /* [batch][h_kv]                         */
    const uint8_t*  q_codes;      /* [Tq][h_q][64]                         */
    const uint8_t*  q_scales;     /* [Tq][h_q][8]                          */
    const float*    q_tscale;     /* [batch][h_q]                          */
    const void*     v_aux;        /* with ORC_PV_BF16 / ORC_PV_NVFP4 in flags */
    int64_t         num_pages;    /* cache capacity in pages (plane size of v_aux) */
} orc_cache;

/* Causal prefill over the paged cache for selected rows.
 * cu_seqlens [batch+1] indexes q tokens; q_start [batch] is the absolute
 * position of each sequence's first query.  Item n is query row item_row[n]
 * (0-based within its sequence) of sequence item_b[n], head item_h[n].
 * Outputs bf16 [n][128] and optionally FP64 [n][128].                      */
int orc_prefill(const orc_cache* c, const int32_t* cu_seqlens, const int32_t* q_start,
                int64_t n_items, const int32_t* item_b, const int32_t* item_row,
                const int32_t* item_h, uint16_t* out_bf16, double* out_f64);

/* Split-KV decode: one query token per sequence (q rows indexed by b), all
 * kv_len[b] keys, partitions of partition_tokens keys merged by LSE.      */
int orc_decode(const orc_cache* c, int32_t partition_tokens,
               int64_t n_items, const int32_t* item_b, const int32_t* item_h,
               uint16_t* out_bf16, double* out_f64);

/* MXFP4 row (the 32-element E8M0 variant Eq. 1 names as the MX format):
 * per 32-channel block, X = 2^e with e = floor(log2 amax) - 2 (the largest
 * E2M1 exponent is 2), clamped to [-127, 127] (e = -127 when amax = 0);
 * code = E2M1(x / X), round to nearest even, saturating at 6.  Scale bytes
 * 0..3 hold e + 127, bytes 4..7 are zero.  Parity unpinned beyond the codec
 * pins: the paper gives no MXFP4 example. */
void orc_mxfp4_row(const float* xc, uint8_t* codes64, uint8_t* scales8);
void orc_mxfp4_dequant_row(const uint8_t* codes64, const uint8_t* scales8, double* out);

/* Dequantize one NVFP4 row (128 values) to FP64: t * dec(s_g) * dec(q). */
void orc_nvfp4_dequant_row(const uint8_t* codes64, const uint8_t* scales8, double t,
                           double* out);

int orc_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
