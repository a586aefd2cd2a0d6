/*
 * Softmax ablation, built as libmpfa_ablate.so for the benchmark's
 * characterization leg (the product library libmpfa.so does not contain it).
 * The library holds the product kernels plus two ablated builds of the causal
 * prefill (compensation as accumulator input, FP8 P and V, NVFP4 or MXFP4
 * Q/K); the cost of a softmax stage is the time difference between levels
 * (Sec. 3.2, Fig. 3c).  Outputs of an ablated level are meaningless by design.
 */
#ifndef MPFA_ABLATE_H
#define MPFA_ABLATE_H

#include "mpfa.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Selects what later mpfa_prefill calls of this library run when they take
 * the method's path (MPFA_SMOOTH, no seed or PV characterization flags):
 *   0  the product kernel;
 *   1  P = its exponent argument (no exp2);
 *   2  as 1, and no row maximum, row sum or O rescale.
 * Host state of the process (not per stream or device); returns 0, or 1 for a
 * level outside 0..2 (the level is then unchanged).
 */
int mpfa_ablation_set_level(int level);

#ifdef __cplusplus
}
#endif

#endif /* MPFA_ABLATE_H */
