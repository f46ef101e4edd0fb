// Measurement aid, not part of the method: the plain in-place read-modify-write ceiling of a
// buffer. Every 16-byte vector is XORed with a 32-bit key replicated four times, in the
// streaming shape of the bf16 perturb sweep and with no other work: each wave walks a chunk
// of up to 32 KiB in steps of 2 KiB (two rows of 64 lanes x 16 bytes, non-temporal loads and
// stores) with the loads of the next two steps in flight, grid-stride over chunks with
// 65,536 workgroups of 256 threads, one workgroup per CU at a time (dynamic LDS). Two calls
// with the same key restore the buffer exactly.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kBlock = 256;
constexpr uint64_t kStepVecs = 128;      // 2 KiB per wave step
constexpr uint64_t kChunkSteps = 16;     // 32 KiB per wave chunk
constexpr uint32_t kGrid = 65536;
constexpr size_t kOnePerCuLds = 96 * 1024;

__device__ __forceinline__ void load_step(u32x4 (&d)[2], const u32x4* q) {
  d[0] = __builtin_nontemporal_load(q);
  d[1] = __builtin_nontemporal_load(q + 64);
}
__device__ __forceinline__ void store_step(u32x4* q, const u32x4 (&d)[2], u32x4 k) {
  __builtin_nontemporal_store(d[0] ^ k, q);
  __builtin_nontemporal_store(d[1] ^ k, q + 64);
}

__global__ __launch_bounds__(kBlock) void xor_sweep(u32x4* p, uint64_t n_vecs, uint32_t key) {
  extern __shared__ uint32_t occupancy_pad[];
  if (key == 0 && n_vecs == 0) occupancy_pad[threadIdx.x] = 0;  // never taken (n_vecs > 0)
  const u32x4 k = {key, key, key, key};
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t n_waves = gridDim.x * (kBlock / 64);
  // 32-bit step and chunk indices (the host keeps a call below 2^31 chunks): the loop
  // control stays on the scalar unit
  const uint32_t n_steps = static_cast<uint32_t>(n_vecs / kStepVecs);
  const uint32_t n_chunks = (n_steps + kChunkSteps - 1) / kChunkSteps;
  for (uint32_t c = blockIdx.x * (kBlock / 64) + wave; c < n_chunks; c += n_waves) {
    const uint32_t s0 = c * kChunkSteps, s1 = s0 + kChunkSteps < n_steps ? s0 + kChunkSteps : n_steps;
    u32x4* q = p + static_cast<uint64_t>(s0) * kStepVecs + lane;
    // rotating register sets with the loads of the next two steps in flight, and one full
    // step run before the loop so that the loop is entered with the same memory operations
    // outstanding as on its back edge (as the perturb sweep)
    u32x4 x[2], y[2], z[2];
    auto prefetch2 = [&](u32x4 (&d)[2]) {
      load_step(d, q + 2 * kStepVecs);
      __builtin_amdgcn_sched_barrier(0);
    };
    auto work = [&](const u32x4 (&d)[2]) {
      store_step(q, d, k);
      q += kStepVecs;
    };
    auto step3 = [&]() {
      prefetch2(z);
      work(x);
      prefetch2(x);
      work(y);
      prefetch2(y);
      work(z);
    };
    auto last = [&](uint32_t left) {  // 2 to 4 steps left, x and y requested
      if (left >= 3) {
        prefetch2(z);
        work(x);
        if (left == 4) {
          prefetch2(x);
          work(y);
          work(z);
          work(x);
        } else {
          work(y);
          work(z);
        }
      } else {
        work(x);
        work(y);
      }
    };
    load_step(x, q);
    uint32_t s = s0;
    if (s + 4 < s1) {
      load_step(y, q + kStepVecs);
      step3();
      s += 3;
      for (; s + 4 < s1; s += 3) step3();
      last(s1 - s);
    } else if (s + 1 < s1) {
      load_step(y, q + kStepVecs);
      last(s1 - s);
    } else {
      work(x);
    }
  }
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t v = static_cast<uint64_t>(n_steps) * kStepVecs + static_cast<uint64_t>(blockIdx.x) * kBlock +
                    threadIdx.x;
       v < n_vecs; v += stride)
    p[v] = p[v] ^ k;
}

}  // namespace

// 0 on success; -1 for a null pointer with bytes > 0; -2 when p is not 16-byte aligned,
// bytes is not a multiple of 16 or reaches 2^46; -4 when the launch fails. Asynchronous on
// `stream`.
extern "C" int zo_calib_rmw(void* p, uint64_t bytes, uint32_t key, void* stream) {
  if (bytes == 0) return 0;
  if (p == nullptr) return -1;
  if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0 || (bytes & 15u) != 0) return -2;
  if (bytes >= (1ull << 46)) return -2;  // 2^31 chunks of 32 KiB
  const uint64_t n_vecs = bytes / 16;
  const uint64_t chunks = (n_vecs / kStepVecs + kChunkSteps - 1) / kChunkSteps;
  uint64_t blocks = (chunks + 3) / 4;
  if (blocks < 1) blocks = 1;
  if (blocks > kGrid) blocks = kGrid;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(xor_sweep), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(kOnePerCuLds));
  hipLaunchKernelGGL(xor_sweep, dim3(static_cast<uint32_t>(blocks)), dim3(kBlock), kOnePerCuLds,
                     static_cast<hipStream_t>(stream), static_cast<u32x4*>(p), n_vecs, key);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
