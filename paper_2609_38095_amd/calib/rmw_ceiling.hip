// Measurement aid, not part of the method: the plain in-place read-modify-write ceiling of a
// buffer. Every 16-byte vector is XORed with a 32-bit key replicated four times, with no other
// work, by the sweeps' own streaming loop (zo_stream.h) over the buffer taken as bf16 weights:
// row groups of two rows of 64 lanes x 16 bytes, non-temporal loads and stores, chunks of up
// to 32 KiB per wave with the loads of the next two groups in flight, one workgroup of 256
// threads per CU at a time (dynamic LDS), and the sweeps' launch plan (zo_plan.cpp). Shapes:
// grid-stride over up to 65,536 workgroups or one chunk per wave, unpaced or paced (at four
// outstanding memory operations with two groups in flight, six with three), as the sweeps are
// launched. Two calls with the same key restore the buffer exactly.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "zo_plan.h"
#include "zo_stream.h"

namespace {

using namespace zo;

template <int AHEAD, int PACE>
__global__ __launch_bounds__(kBlock) void xor_sweep(Plans<1> ps, uint32_t key) {
  extern __shared__ uint32_t occupancy_pad[];  // dynamic LDS only limits workgroups per CU
  if (ps.count == 0xFFFFFFFFu) occupancy_pad[threadIdx.x] = 0;  // never taken (count is 1)
  const u32x4 k = {key, key, key, key};
  constexpr int R = GroupShape<BF16>::kRows;
  for_each_group<BF16, AHEAD, 1, PACE, kBlock, 1>(
      ps,
      [&](uint64_t, u32x4 (&d)[R], uint32_t) {
#pragma unroll
        for (int u = 0; u < R; ++u) {
          // the empty asm makes the XOR opaque: with a body this light the compiler otherwise
          // keeps the loop's rotating register sets in scratch memory
          u32x4 t = d[u] ^ k;
          asm volatile("" : "+v"(t));
          d[u] = t;
        }
      },
      []() {});
  // head and tail elements: element g of the buffer is XORed with the key's low 16 bits
  // (g even) or high 16 bits (g odd), as the 16-byte XOR does
  for_each_edge<1, kBlock>(ps, [&](const Plan& pl, uint64_t t) {
    uint16_t* p = reinterpret_cast<uint16_t*>(pl.base);
    for (uint64_t g = t * kTile; g < (t + 1) * kTile; ++g)
      if (g >= pl.lo && g < pl.hi) p[g - pl.lo] ^= static_cast<uint16_t>(g & 1 ? key >> 16 : key);
  });
}

}  // namespace

// shape: bit 0 one chunk per wave, bit 1 paced, bit 2 three groups in flight instead of two.
// 0 on success; -1 for a null pointer with bytes > 0; -2 when p is not 16-byte aligned, bytes
// is not a multiple of 16 or reaches 2^41, or shape has other bits; -4 when the launch fails.
// Asynchronous on `stream`.
extern "C" int zo_calib_rmw_shape(void* p, uint64_t bytes, uint32_t key, uint32_t shape, void* stream) {
  if (bytes == 0) return 0;
  if (p == nullptr) return -1;
  if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0 || (bytes & 15u) != 0) return -2;
  if (bytes / 2 >= ZO_N_MAX) return -2;
  if (shape & ~7u) return -2;
  const bool one_chunk_per_wave = shape & 1u, paced = shape & 2u;
  const Shape sh{static_cast<uint32_t>(kMaxChunkBytes / (kGroupElems * 2)), 1, one_chunk_per_wave ? 1u : 0u};
  Plans<1> ps{};
  ps.chunk_groups = sh.chunk_groups;
  add_plan(ps, make_plan(p, 0, bytes / 2, 2, sh.chunk_groups), 2, streams_per_block(sh));
  const size_t pad = occupancy_lds(sh.blocks_per_cu, 0);
  const bool three = shape & 4u;
  // paced: the step's own prefetch and the previous step's last stores stay outstanding
  auto kernel = three ? (paced ? xor_sweep<3, 6> : xor_sweep<3, 0>) : (paced ? xor_sweep<2, 4> : xor_sweep<2, 0>);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(pad));
  (void)hipGetLastError();
  hipLaunchKernelGGL(kernel, dim3(plans_grid(ps, sh)), dim3(kBlock), pad, static_cast<hipStream_t>(stream), ps,
                     key);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" int zo_calib_rmw(void* p, uint64_t bytes, uint32_t key, void* stream) {
  return zo_calib_rmw_shape(p, bytes, key, 0, stream);
}
