/*
 * sphinx_prof.h -- measurement aids of libsphinx (outside the method).
 *
 * Per-kernel-class timing with HIP events, and a calibration kernel for the
 * achievable dense bf16 MFMA rate.  Neither takes part in the
 * selective-refinement step declared in sphinx.h; they exist so that a
 * benchmark can attribute a step's time to its kernels and read the kernels'
 * rates against the rate the matrix cores sustain.
 */
#ifndef SPHINX_PROF_H
#define SPHINX_PROF_H

#include "sphinx.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Profiling aid (outside the method).  sphinx_timing_enable(classes) takes a
 * bit mask of kernel classes (bit k = class k; 0 turns timing off; bits at or
 * above SPHINX_K_COUNT are SPHINX_E_INVALID).  While a class is enabled, every
 * launch of it is bracketed by two HIP events recorded on the stream of the
 * launch; sphinx_timing_read waits for the recorded events and returns the
 * number of launches and their summed GPU time since timing was last enabled
 * (a non-zero mask resets the sums).  Bracketing only the classes of interest
 * keeps the events away from the other launches.  Events are created on first
 * use and reused; nothing is allocated on the device.  The timing state is
 * process-wide and guarded by a mutex. */
typedef SPHINX_ENUM {
  SPHINX_K_SELECT = 0, /* mask + compaction (three kernels, one bracket) */
  SPHINX_K_GATHER,
  SPHINX_K_COND,       /* timestep/adaLN conditioning, position tables, token metadata */
  SPHINX_K_EMBED,
  SPHINX_K_LN,         /* adaLN LayerNorm before QKV and MLP1 */
  SPHINX_K_GEMM_QKV,
  SPHINX_K_ATTENTION,
  SPHINX_K_GEMM_OUT,
  SPHINX_K_GEMM_MLP1,
  SPHINX_K_GEMM_MLP2,
  SPHINX_K_FINAL,      /* final LayerNorm + projection + DDIM update */
  SPHINX_K_SCATTER,
  SPHINX_K_KV_STORE,   /* latent cache store of the forwarded rows' keys and values */
  SPHINX_K_FRONTEND,   /* mask front-end (five kernels, one bracket) */
  SPHINX_K_COUNT
} sphinx_kernel_class;

sphinx_status sphinx_timing_enable(int32_t classes);
sphinx_status sphinx_timing_read(sphinx_kernel_class k, int64_t* launches, double* total_ms);

/* Calibration aid (outside the method): the achievable dense bf16 MFMA rate.
 * Enqueues SPHINX_PEAK_BLOCKS workgroups of 4 waves; each wave runs `iters`
 * rounds of four independent v_mfma_f32_32x32x16_bf16 chains (4 * 32768 FLOP
 * per round) and writes one checksum float per workgroup to `out` (dev float
 * [SPHINX_PEAK_BLOCKS], caller-owned).  FLOPs per call:
 * SPHINX_PEAK_BLOCKS * 4 * iters * 4 * 32768; the caller times the call on
 * `stream`.  iters must lie in [1, 2^24].  operands selects the data the
 * MFMAs multiply, since the sustained rate depends on it (the chip lowers its
 * clock as the operand bits toggle more):
 *   SPHINX_PEAK_CONSTANT: small constants, the same every round (best case);
 *   SPHINX_PEAK_RANDOM:   hashed random bf16 in [-2, 2), eight operand pairs
 *                         in rotation (closer to real activations).
 * Any other value: SPHINX_E_INVALID. */
#define SPHINX_PEAK_BLOCKS 2048
#define SPHINX_PEAK_CONSTANT 0
#define SPHINX_PEAK_RANDOM 1
sphinx_status sphinx_peak_mfma(int32_t iters, int32_t operands, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPHINX_PROF_H */
