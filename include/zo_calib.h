/* zo_calib.h - measurement aid shipped beside libzo (libzo_calib.so); not part of the method.
 *
 * The probe sweeps are bound by HBM read-modify-write bandwidth, which on MI355X depends on
 * the access pattern and, for some patterns, on where a buffer sits physically. zo_calib_rmw
 * gives the plain ceiling of a given buffer in the sweeps' own access pattern, so a sweep's
 * rate can be reported as a fraction of it as well as of the nominal 8 TB/s.
 */
#ifndef ZO_CALIB_H
#define ZO_CALIB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* XOR every 16-byte vector of p[0 .. bytes) in place with `key` replicated four times:
 * one read and one write of every byte, by the sweeps' own streaming loop and launch plan
 * (the buffer taken as bf16 weights: each wave walks up to 32 KiB in 2 KiB row groups with
 * the next two groups' loads in flight, non-temporal loads and stores, one workgroup of 256
 * threads per CU at a time, grid-stride over up to 65,536 workgroups) and no other work. Two
 * calls with the same key restore the buffer bit for bit.
 *   p      caller-owned device memory, 16-byte aligned; bytes a multiple of 16, below 2^41.
 *   stream hipStream_t (NULL = default stream); the call is asynchronous on it.
 * Returns 0; -1 for p == NULL with bytes > 0; -2 for misalignment or a size that is not a
 * multiple of 16 or too large (nothing launched); -4 when the launch fails. bytes == 0 is a
 * no-op. */
int zo_calib_rmw(void* p, uint64_t bytes, uint32_t key, void* stream);

/* zo_calib_rmw in another launch shape, so that the ceiling can be taken as the fastest of
 * several: shape bit 0 = one 32 KiB chunk per wave (a grid sized to the buffer instead of
 * grid-stride), bit 1 = paced (each step of the loop first waits until at most four memory
 * operations of the wave are outstanding, six with three groups in flight), bit 2 = the loads
 * of three row groups in flight instead of two. shape 0 is zo_calib_rmw. Returns as zo_calib_rmw, and -2 also for shape
 * bits above bit 2 (nothing launched). */
int zo_calib_rmw_shape(void* p, uint64_t bytes, uint32_t key, uint32_t shape, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ZO_CALIB_H */
