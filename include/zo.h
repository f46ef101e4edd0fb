/*
 * zo.h -- C ABI of libzo: the probe regenerate-and-apply sweep of 1.5-SPSA on gfx950.
 *
 * 1.5-SPSA ("Probe-Space Preconditioning for Fast and Stable Zero-Order Training")
 * estimates a descent direction from antithetic loss pairs L(theta +- eps z_k) along
 * Rademacher probes z_k plus one clean loss L(theta), and weights each probe by its
 * measured curvature (section 4.1, Eq. 3 and 4; section 4.2, Eq. 5 and 6; Algorithm 1).
 * The probes are never stored: every sweep regenerates z_k from (seed, step, k, element
 * index) with a counter-based generator, 8 probe signs per byte (section 4.3).
 *
 * Probe definition (shared by every call below):
 *   element i (a 64-bit global index) belongs to tile t = i / 16; probe k belongs to
 *   group g = k / 8. The tile's block is Philox4x32-10 (Salmon et al., SC'11) with
 *   counter (t mod 2^32, t / 2^32, step, g) and key (seed mod 2^32, seed / 2^32), four
 *   32-bit words x0..x3. Element i's byte is byte (i mod 4) of word x_((i mod 16) / 4);
 *   z_k[i] = +1 if bit (k mod 8) of that byte is set, else -1 (appendix F's convention).
 *
 * Conventions for every call:
 *   - params: caller-owned device memory, a contiguous flat array of n elements of the
 *     given dtype, aligned to the element size. The library never allocates, frees or
 *     retains it; it must stay valid until the stream work has finished.
 *   - offset: the global element index of params[0], so a shard or window of a larger
 *     parameter vector regenerates the same probe values as the whole vector would.
 *     offset + n must be below 2^64.
 *   - stream: a hipStream_t (NULL = the default stream). Device work is enqueued on it
 *     and the call returns without waiting; faults surface at the caller's next
 *     synchronisation. Host arguments (coefficient arrays) are copied before return.
 *   - device: params (every segment's) and stream belong to the calling thread's current
 *     HIP device, on which the kernels are launched.
 *   - Errors: every argument is validated before anything is launched; on ZO_ERR_NULL,
 *     ZO_ERR_ARG or ZO_ERR_NONFINITE nothing was enqueued and no output was written.
 *     ZO_ERR_HIP reports a launch the runtime refused (for the segment calls, earlier
 *     batches of the same call may already be enqueued). n = 0 (or K = 0) is a successful
 *     no-op.
 *   - No global state is kept between calls except an optional launch-width override
 *     (zo_set_max_blocks); calls on different streams may run concurrently on disjoint
 *     parameter memory. The library allocates no device memory.
 */
#ifndef ZO_H_
#define ZO_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { ZO_F32 = 0, ZO_BF16 = 1 } zo_dtype;

enum {
  ZO_OK = 0,
  ZO_ERR_NULL = -1,      /* a required pointer is NULL */
  ZO_ERR_ARG = -2,       /* bad dtype, misalignment, K or n out of range, index overflow */
  ZO_ERR_NONFINITE = -3, /* a non-finite eps, lr, loss or coefficient */
  ZO_ERR_HIP = -4        /* the HIP runtime refused the launch */
};

/* Most probes one zo_update call applies (coefficients travel as kernel arguments, 4 KiB). */
#define ZO_K_MAX 1024u

/* Every call and every segment covers fewer than ZO_N_MAX = 2^40 elements (2 TiB of bf16,
 * more than any one device holds); larger n is ZO_ERR_ARG. */
#define ZO_N_MAX (1ull << 40)

/* One tensor of a model's parameters, for the *_segments calls: `params` is caller-owned
 * device memory (aligned to the element size, on the device the stream belongs to) holding
 * n elements whose global element indices are offset .. offset + n - 1. */
typedef struct {
  void* params;
  uint64_t offset;
  uint64_t n;
} zo_segment;

/*
 * zo_perturb -- theta[i] <- theta[i] + eps * z_k[offset + i], for i in [0, n).
 * Algorithm 1 applies each probe three times around its two perturbed forward passes,
 * with eps = +e, then -2e, then +e (restoring theta up to rounding).
 * Arithmetic: one IEEE fp32 addition (bf16 weights widened exactly, the sum rounded back
 * to bf16 to nearest-even). The result is bit-exact and independent of launch shape.
 * Errors: ZO_ERR_NULL (params NULL with n > 0), ZO_ERR_ARG (dtype, alignment, index
 * overflow, n >= ZO_N_MAX), ZO_ERR_NONFINITE (eps), ZO_ERR_HIP.
 */
int zo_perturb(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed,
               uint32_t step, uint32_t k, float eps, void* stream);

/*
 * zo_probe_coeffs -- host function: per-probe update coefficients c[K] from the losses.
 *   curvature (section 4.1, Eq. 3):   chat_k = (L_plus[k] - 2 L_clean + L_minus[k]) / eps^2
 *   weight    (section 4.1, Eq. 4):   w_k = 1 / max(lambda_reg, |chat_k|^alpha)
 *   coefficient (Eq. 5/6, Alg. 1):    c_k = w_k (L_plus[k] - L_minus[k]) / (2 K eps)
 * so that zo_update with lr = eps applies Algorithm 1's gamma_k = (1/2n)(L+ - L-) w_k.
 * zo_probe_coeffs uses the paper's alpha = 0.1 and lambda_reg = 1.
 * Arithmetic is IEEE float64 in exactly this order: d2 = (L+ - 2*L0) + L-;
 * chat = d2/(eps*eps); a = pow(|chat|, alpha); den = a > lambda_reg ? a : lambda_reg;
 * w = 1/den; c64 = ((L+ - L-)*w)/((2*K)*eps); c = (float)c64 (nearest-even).
 * Inputs are host arrays of K doubles; outputs are host arrays of K entries, each
 * optional (NULL) in the _ex form. Never touches the GPU.
 * Errors: ZO_ERR_NULL (loss arrays or c_out NULL), ZO_ERR_ARG (K = 0, eps <= 0,
 * alpha outside [0, 1], lambda_reg <= 0), ZO_ERR_NONFINITE (any non-finite input).
 * Outputs are written only on success.
 */
int zo_probe_coeffs(const double* L_plus, const double* L_minus, uint32_t K, double L_clean,
                    double eps, float* c_out);
int zo_probe_coeffs_ex(const double* L_plus, const double* L_minus, uint32_t K, double L_clean,
                       double eps, double alpha, double lambda_reg, float* c_out,
                       double* c64_out, double* curv_out, double* w_out);

/*
 * zo_update -- theta[i] <- theta[i] - lr * sum_{k<K} c[k] z_k[i], for global i in [0, n).
 * The fused form of section 4.2 (Eq. 6, Delta theta = -eta Z W Delta l) and of
 * Algorithm 1's per-probe loop: one read and one write of theta for all K probes, which
 * are regenerated in registers. c: host array of K floats (from zo_probe_coeffs).
 * Arithmetic: per element, s = sum over the probe groups of fl(lr * t_g) in fp32, where t_g is
 * the pairwise fp32 sum of the element's 8 signed c[k] of group g (sequential across groups
 * within runs of 8 groups, compensated across runs); theta - s in fp32, then one rounding
 * to bf16 for bf16 weights. With K = 1 this equals zo_perturb(k = 0,
 * eps = -fl(lr * c[0])) bit for bit.
 * Errors: ZO_ERR_NULL (params NULL with n > 0, c NULL with K > 0), ZO_ERR_ARG (dtype,
 * alignment, K > ZO_K_MAX, k_base + K > 2^32), ZO_ERR_NONFINITE (lr or any c[k]), ZO_ERR_HIP.
 * Cost: one read and one write of theta; above about 16 probes (bf16) the sweep is bound by
 * the probe generator and the table arithmetic (VALU) rather than by HBM.
 */
int zo_update(void* params, zo_dtype dtype, uint64_t n, uint64_t seed, uint32_t step,
              uint32_t K, const float* c, float lr, void* stream);

/*
 * zo_update_ex -- zo_update over global elements [offset, offset + n) for probes
 * k_base .. k_base + K - 1 (c[j] belongs to probe k_base + j). A shard of a larger
 * vector passes its offset; more than ZO_K_MAX probes are applied as several calls with
 * increasing k_base (each call rounds theta once).
 */
int zo_update_ex(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed,
                 uint32_t step, uint32_t k_base, uint32_t K, const float* c, float lr,
                 void* stream);

/*
 * zo_perturb2 -- theta[i] <- theta[i] + (eps_a z_{k_a}[offset+i] + eps_b z_{k_b}[offset+i]),
 * one sweep. On one device Algorithm 1's restore of probe k (+eps) and the +eps of probe
 * k + 1 are consecutive applications; this applies the pair in one pass, so a step needs
 * 2K + 1 sweeps instead of 3K + 1. Arithmetic: d = fl32(eps_a z_a + eps_b z_b) (exact when
 * |eps_a| = |eps_b|), one fp32 addition theta + d, then one rounding to bf16 for bf16
 * weights; bit-exact and independent of launch shape. k_a may equal k_b; eps_b = 0 gives
 * exactly zo_perturb(k_a, eps_a).
 * Errors: as zo_perturb (ZO_ERR_NONFINITE for a non-finite eps_a or eps_b).
 */
int zo_perturb2(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed,
                uint32_t step, uint32_t k_a, float eps_a, uint32_t k_b, float eps_b, void* stream);

/*
 * zo_update_restore -- theta[i] <- theta[i] + eps_restore z_{k_restore}[offset+i]
 *                                  - lr * sum_j c[j] z_{k_base+j}[offset+i], one sweep:
 * the last probe's restore merged with the fused update (Algorithm 1's final +eps and its
 * rank-0 update loop; section 4.2, Eq. 6). Arithmetic per element in fp32, s as in
 * zo_update: when k_restore lies in one of the update's probe groups (8 j .. 8 j + 7 for a
 * group j that holds one of the K probes; Algorithm 1 restores probe k_base + K - 1), that
 * group's term fl(lr * t_g) becomes fl(fl(lr * t_g) - eps_restore z) and the result is
 * theta - s; otherwise t = fl(theta + eps_restore z), then t - s. Then one rounding to bf16
 * for bf16 weights. eps_restore = 0 gives zo_update_ex's result bit for bit.
 * Errors: as zo_update_ex (ZO_ERR_NONFINITE also for a non-finite eps_restore). With K = 0
 * it applies the restore alone.
 */
int zo_update_restore(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed,
                      uint32_t step, uint32_t k_base, uint32_t K, const float* c, float lr,
                      uint32_t k_restore, float eps_restore, void* stream);

/*
 * zo_perturb_segments -- zo_perturb2 over a list of separate tensors (a model that keeps
 * its parameters in separate allocations rather than one flat buffer): for every segment s,
 * theta_s[i] <- theta_s[i] + (eps_a z_{k_a} + eps_b z_{k_b})[offset_s + i]. eps_b = 0 is the
 * one-probe zo_perturb. Each element's result is exactly what zo_perturb / zo_perturb2 give
 * for that tensor alone. segs: host array of n_segs entries, read during the call.
 * Segments with n = 0 are skipped; the global index ranges may be in any order but the
 * segments' memory must not overlap. The tensors are swept in launches of up to 64
 * segments each (one sweep's worth of HBM traffic in total).
 * Errors: ZO_ERR_NULL (segs NULL with n_segs > 0, a segment's params NULL with n > 0),
 * ZO_ERR_ARG (dtype, a misaligned segment, an index range reaching 2^64, a segment of
 * ZO_N_MAX elements or more, overlapping segments), ZO_ERR_NONFINITE, all before anything is launched; ZO_ERR_HIP if a launch
 * fails, in which case earlier batches may already be enqueued.
 */
int zo_perturb_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype, uint64_t seed,
                        uint32_t step, uint32_t k_a, float eps_a, uint32_t k_b, float eps_b,
                        void* stream);

/*
 * zo_update_segments -- zo_update_restore over a list of separate tensors (see
 * zo_perturb_segments for the segment rules): theta_s <- theta_s + eps_restore z_{k_restore}
 * - lr * sum_j c[j] z_{k_base+j}, each element as zo_update_restore computes it for that
 * tensor alone; eps_restore = 0 is zo_update_ex. Errors: as zo_perturb_segments, plus those
 * of zo_update_ex for K, k_base and c.
 */
int zo_update_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype, uint64_t seed,
                       uint32_t step, uint32_t k_base, uint32_t K, const float* c, float lr,
                       uint32_t k_restore, float eps_restore, void* stream);

/*
 * zo_gen_bits -- writes the raw 16-byte probe block of each tile tile_begin ..
 * tile_begin + n_tiles - 1 for probe group `group` (probes 8*group .. 8*group+7) to
 * out_dev (device memory, 16 * n_tiles bytes, caller-owned). Exposes the generator for
 * bit-exact checks; the sweeps never store probes.
 * Errors: ZO_ERR_NULL (out_dev NULL with n_tiles > 0), ZO_ERR_ARG (out_dev not 16-byte
 * aligned, or tile indices reaching 2^60, the tile of element index 2^64), ZO_ERR_HIP.
 */
int zo_gen_bits(uint8_t* out_dev, uint64_t tile_begin, uint64_t n_tiles, uint64_t seed,
                uint32_t step, uint32_t group, void* stream);

/* zo_strerror -- static description of a status code. */
const char* zo_strerror(int status);

/*
 * zo_set_max_blocks -- a test hook: caps the number of workgroups of every later sweep
 * launch in the process (0 restores the default shapes), so that tests can check that
 * results do not depend on the grid. Results never depend on it. The value is stored
 * atomically (a launch on another thread sees the old or the new cap, never a mix), but it
 * is process-wide: it changes the launches of every caller, on every stream, until reset.
 */
void zo_set_max_blocks(uint32_t max_blocks);

/* zo_version -- library version string. */
const char* zo_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ZO_H_ */
