/*
 * Measurement probes, built as libmpfa_probe.so for the benchmark (the product
 * library libmpfa.so does not contain them): the achievable matrix-core rate of each
 * MFMA form the attention kernels use, and the achievable HBM read rate, both
 * measured on the device itself.  They serve as the second denominator of the
 * kernels' roofline fractions, next to the published peaks (dense MFMA: FP16
 * 2.5 PFLOP/s, FP8 5.0, FP4 10.1; HBM 8 TB/s).
 *
 * Both calls validate on the host before any HIP call (MPFA_ERR_INVALID),
 * launch one kernel on `stream`, return without synchronizing, and allocate
 * nothing.  The caller times them (HIP events on the same stream).
 */
#ifndef MPFA_PROBE_H
#define MPFA_PROBE_H

#include "mpfa.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
    MPFA_PROBE_MFMA_F16 = 0,   /* v_mfma_f32_16x16x32_f16: 16 x 16 x 32, 16384 FLOP      */
    MPFA_PROBE_MFMA_FP8 = 1,   /* v_mfma_scale_f32_16x16x128_f8f6f4, E4M3 x E4M3, 65536 FLOP */
    MPFA_PROBE_MFMA_FP4 = 2    /* the same instruction, E2M1 x E2M1, 65536 FLOP          */
};

enum {
    MPFA_PROBE_READ_VGPR = 0,  /* 16-byte global loads into registers                  */
    MPFA_PROBE_READ_LDS = 1    /* 16-byte direct global -> LDS loads (global_load_lds)  */
};

/*
 * MFMA issue rate.  `blocks` workgroups of 256 threads (4 waves) each run
 * `iters` rounds of 8 independent MFMAs of form `kind` per wave.  Every
 * operand register of A holds the 32-bit word `pa`, every one of B holds `pb`
 * (FP4: the four registers of the 32 E2M1 codes), block scales are 2^0.
 * sink: device float[blocks * 256]; lane i of block b writes the sum of its 32
 * accumulator values there.  With A and B all ones (pa = pb = 0x3C003C00 for
 * FP16, 0x38383838 for E4M3, 0x22222222 for E2M1) that sum is exactly
 * 32 * K * iters, K = 32 (F16) or 128 (FP8, FP4), for iters * K < 2^24.
 * FLOP per launch: blocks * 4 * iters * 8 * (2 * 16 * 16 * K).
 * Errors: MPFA_ERR_INVALID for an unknown kind, iters < 1, blocks outside
 * [1, 2^20] or a null sink; MPFA_ERR_HIP if the launch fails.
 */
mpfa_status mpfa_probe_mfma(int32_t kind, int32_t iters, int32_t blocks, uint32_t pa, uint32_t pb,
                            float* sink, mpfa_stream_t stream);

/*
 * HBM read rate.  Reads the `bytes` bytes at device address `src` once, as
 * 16-byte words: workgroup b streams the contiguous b-th of `blocks` equal
 * shares, in rounds of 8 words per thread (mode READ_VGPR into registers;
 * READ_LDS through direct global -> LDS loads into a 32 KB slab per workgroup,
 * read back by the same lane).  sink: device uint32[blocks * 256]; each
 * thread writes the XOR of the 32-bit words it read, so the XOR of the whole
 * sink equals the XOR of all words of the buffer.
 * Errors: MPFA_ERR_INVALID for an unknown mode, a null or unaligned (16-byte)
 * src, a null sink, blocks outside [1, 2^20], or bytes not a positive multiple
 * of blocks * 256 * 8 * 16; MPFA_ERR_HIP if the launch fails.
 */
mpfa_status mpfa_probe_read(int32_t mode, const void* src, int64_t bytes, int32_t blocks, uint32_t* sink,
                            mpfa_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MPFA_PROBE_H */
