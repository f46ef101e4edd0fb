// Measurement aid, not part of the method: the plain in-place read-modify-write ceiling of a
// buffer. Every 16-byte vector is XORed with a 32-bit key replicated four times, with the
// sweep kernels' memory shape (one wave moves 1 KiB per instruction, four instructions per
// chunk, non-temporal loads and stores, grid-stride over chunks, 65,536 workgroups of 256
// threads) and no other work. Two calls with the same key restore the buffer exactly.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kBlock = 256;
constexpr uint64_t kChunkVecs = 256;  // 4 KiB per wave
constexpr uint32_t kGrid = 65536;

__global__ __launch_bounds__(kBlock) void xor_sweep(u32x4* p, uint64_t n_vecs, uint32_t key) {
  const u32x4 k = {key, key, key, key};
  const uint32_t lane = threadIdx.x & 63u;
  const uint64_t n_waves = static_cast<uint64_t>(gridDim.x) * (kBlock / 64);
  const uint64_t n_chunks = n_vecs / kChunkVecs;
  for (uint64_t c = static_cast<uint64_t>(blockIdx.x) * (kBlock / 64) + (threadIdx.x >> 6); c < n_chunks;
       c += n_waves) {
    u32x4* q = p + c * kChunkVecs + lane;
    u32x4 d[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) d[u] = __builtin_nontemporal_load(q + 64 * u);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(d[u] ^ k, q + 64 * u);
  }
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t v = n_chunks * kChunkVecs + static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; v < n_vecs;
       v += stride)
    p[v] = p[v] ^ k;
}

}  // namespace

// 0 on success; -1 for a null pointer with bytes > 0; -2 when p is not 16-byte aligned or
// bytes is not a multiple of 16; -4 when the launch fails. Asynchronous on `stream`.
extern "C" int zo_calib_rmw(void* p, uint64_t bytes, uint32_t key, void* stream) {
  if (bytes == 0) return 0;
  if (p == nullptr) return -1;
  if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0 || (bytes & 15u) != 0) return -2;
  const uint64_t n_vecs = bytes / 16;
  const uint64_t chunks = n_vecs / kChunkVecs;
  uint64_t blocks = (chunks + 3) / 4;
  if (blocks < 1) blocks = 1;
  if (blocks > kGrid) blocks = kGrid;
  hipLaunchKernelGGL(xor_sweep, dim3(static_cast<uint32_t>(blocks)), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), static_cast<u32x4*>(p), n_vecs, key);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
