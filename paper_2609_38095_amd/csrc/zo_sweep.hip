// Probe regenerate-and-apply sweeps of 1.5-SPSA for gfx950 (CDNA4).
//
// zo_perturb applies theta + eps z_k (Algorithm 1's +eps / -2 eps / +eps applications),
// zo_update applies theta - lr sum_k c_k z_k in one pass (section 4.2, Eq. 6), and
// zo_gen_bits exposes the probe generator. Probes are regenerated in registers from
// (seed, step, k, element index) with Philox4x32-10 (Salmon et al., SC'11), one block per
// 16-element tile and probe group of 8, 8 probe signs per byte (section 4.3); nothing but
// theta touches HBM.
//
// Work decomposition: a persistent grid-stride loop over tiles. A lane owns one tile per
// iteration: 16 elements, i.e. 32 bytes of bf16 or 64 bytes of fp32 moved with 16-byte
// non-temporal loads and stores (theta is streamed once per sweep; nothing is reused).
// The update keeps, per probe group, a 256-entry table in LDS: entry b is the signed sum
// of the group's 8 coefficients selected by the bits of b, so applying 8 probes to an
// element costs one byte extract and one LDS read instead of 8 sign selects.
//
// Built with -ffp-contract=off: every product and sum is rounded as written.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "zo.h"

namespace {

constexpr uint32_t kTile = 16;       // elements per generator block
constexpr uint32_t kBlock = 256;     // threads per workgroup
constexpr uint32_t kDefaultMaxBlocks = 8192;
constexpr int kRounds = 10;

uint32_t g_max_blocks = 0;  // 0: default

// ---------------------------------------------------------------------------------------
// Philox4x32-R: round (x0,x1,x2,x3) -> (hi(M1 x2)^x1^k0, lo(M1 x2), hi(M0 x0)^x3^k1, lo(M0 x0)),
// key bumped by the Weyl constants after each round. The 32x32->64 products map to
// v_mad_u64_u32.
__device__ __forceinline__ uint4 philox4x32(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                            uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * x0;
    const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * x2;
    const uint32_t y0 = static_cast<uint32_t>(p1 >> 32) ^ x1 ^ k0;
    const uint32_t y2 = static_cast<uint32_t>(p0 >> 32) ^ x3 ^ k1;
    x1 = static_cast<uint32_t>(p1);
    x3 = static_cast<uint32_t>(p0);
    x0 = y0;
    x2 = y2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(x0, x1, x2, x3);
}

__device__ __forceinline__ uint4 tile_block(uint64_t t, uint32_t step, uint32_t group, uint32_t k0,
                                            uint32_t k1) {
  return philox4x32(static_cast<uint32_t>(t), static_cast<uint32_t>(t >> 32), step, group, k0, k1);
}

// Byte j (0..15) of a tile's block: byte (j mod 4) of word j / 4.
__device__ __forceinline__ uint32_t block_byte(const uint32_t (&x)[4], int j) {
  return (x[j >> 2] >> (8 * (j & 3))) & 0xFFu;
}

// ---------------------------------------------------------------------------------------
// Storage formats. A tile is moved as 16-byte vectors; values are widened to fp32.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u32x4 ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st_stream(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  const bf16x2 r = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}
__device__ __forceinline__ uint16_t to_bf16(float v) {
  return static_cast<uint16_t>(pack_bf16x2(v, 0.0f) & 0xFFFFu);
}

struct F32 {
  typedef float storage;
  static constexpr uint32_t bytes = 4;
  __device__ static __forceinline__ void load_tile(const storage* p, float (&v)[kTile]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u32x4 w = ld_stream(p + 4 * q);
      v[4 * q + 0] = __uint_as_float(w.x);
      v[4 * q + 1] = __uint_as_float(w.y);
      v[4 * q + 2] = __uint_as_float(w.z);
      v[4 * q + 3] = __uint_as_float(w.w);
    }
  }
  __device__ static __forceinline__ void store_tile(storage* p, const float (&v)[kTile]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u32x4 w = {__float_as_uint(v[4 * q]), __float_as_uint(v[4 * q + 1]),
                       __float_as_uint(v[4 * q + 2]), __float_as_uint(v[4 * q + 3])};
      st_stream(p + 4 * q, w);
    }
  }
  __device__ static __forceinline__ float load1(const storage* p) { return *p; }
  __device__ static __forceinline__ void store1(storage* p, float v) { *p = v; }
};

struct BF16 {
  typedef uint16_t storage;
  static constexpr uint32_t bytes = 2;
  __device__ static __forceinline__ void load_tile(const storage* p, float (&v)[kTile]) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const u32x4 w = ld_stream(p + 8 * q);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        v[8 * q + 2 * m] = __uint_as_float(ws[m] << 16);
        v[8 * q + 2 * m + 1] = __uint_as_float(ws[m] & 0xFFFF0000u);
      }
    }
  }
  __device__ static __forceinline__ void store_tile(storage* p, const float (&v)[kTile]) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const u32x4 w = {pack_bf16x2(v[8 * q + 0], v[8 * q + 1]), pack_bf16x2(v[8 * q + 2], v[8 * q + 3]),
                       pack_bf16x2(v[8 * q + 4], v[8 * q + 5]), pack_bf16x2(v[8 * q + 6], v[8 * q + 7])};
      st_stream(p + 8 * q, w);
    }
  }
  __device__ static __forceinline__ float load1(const storage* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
  __device__ static __forceinline__ void store1(storage* p, float v) { *p = to_bf16(v); }
};

// Range of global elements [lo, hi) covered by a launch and the tiles that touch it.
struct Span {
  uint64_t lo, hi;       // global element indices
  uint64_t t_first;      // first tile
  uint64_t n_tiles;      // tiles touching [lo, hi)
};

// Apply f(j, value) -> value to the elements of tile t inside the span. VEC: the tile's
// storage is 16-byte aligned, so full tiles move as vectors; edge tiles go element-wise.
template <class S, bool VEC, class F>
__device__ __forceinline__ void apply_tile(typename S::storage* params, const Span& sp, uint64_t t, F f) {
  const uint64_t g0 = t * kTile;
  if (VEC && g0 >= sp.lo && g0 + kTile <= sp.hi) {
    typename S::storage* p = params + (g0 - sp.lo);
    float v[kTile];
    S::load_tile(p, v);
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) v[j] = f(j, v[j]);
    S::store_tile(p, v);
  } else {
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) {
      const uint64_t g = g0 + j;
      if (g >= sp.lo && g < sp.hi) {
        typename S::storage* p = params + (g - sp.lo);
        S::store1(p, f(j, S::load1(p)));
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// perturb: theta + eps * z_k. One generator block per tile; bit (k mod 8) of each byte.
template <class S, bool VEC>
__global__ __launch_bounds__(kBlock) void perturb_kernel(typename S::storage* params, Span sp, uint32_t k0,
                                                        uint32_t k1, uint32_t step, uint32_t group,
                                                        uint32_t bit, float eps) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; i < sp.n_tiles; i += stride) {
    const uint64_t t = sp.t_first + i;
    const uint4 r = tile_block(t, step, group, k0, k1);
    const uint32_t x[4] = {r.x, r.y, r.z, r.w};
    apply_tile<S, VEC>(params, sp, t, [&](int j, float v) {
      const bool plus = (block_byte(x, j) >> bit) & 1u;
      return v + (plus ? eps : -eps);
    });
  }
}

// ---------------------------------------------------------------------------------------
// update: theta - lr * sum_k c_k z_k.
struct Coefs {
  float c[ZO_K_MAX];
};

// Sum of the table values of groups [LO, HI) of the launch for the 16 elements of a tile,
// pairwise (a balanced tree over groups). Groups at or past n_groups contribute 0.
template <int LO, int HI, bool GUARD>
__device__ __forceinline__ void group_tree(float (&out)[kTile], const float* tab, uint64_t t, uint32_t step,
                                           uint32_t g_first, uint32_t g_chunk, uint32_t n_groups,
                                           uint32_t k0, uint32_t k1) {
  if constexpr (HI - LO == 1) {
    const uint32_t g = g_chunk + LO;
    if (GUARD && g >= n_groups) {
#pragma unroll
      for (int j = 0; j < (int)kTile; ++j) out[j] = 0.0f;
      return;
    }
    const uint4 r = tile_block(t, step, g_first + g, k0, k1);
    const uint32_t x[4] = {r.x, r.y, r.z, r.w};
    const float* tg = tab + 256u * g;
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) out[j] = tg[block_byte(x, j)];
  } else {
    constexpr int MID = (LO + HI) / 2;
    float a[kTile], b[kTile];
    group_tree<LO, MID, GUARD>(a, tab, t, step, g_first, g_chunk, n_groups, k0, k1);
    group_tree<MID, HI, GUARD>(b, tab, t, step, g_first, g_chunk, n_groups, k0, k1);
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) out[j] = a[j] + b[j];
  }
}

// NG > 0: exactly NG groups (compile time), pairwise over groups.
// NG == 0: any number of groups; chunks of 8 groups summed pairwise, chunks compensated.
template <class S, bool VEC, int NG>
__global__ __launch_bounds__(kBlock) void update_kernel(typename S::storage* params, Span sp, uint32_t k0,
                                                       uint32_t k1, uint32_t step, uint32_t k_base,
                                                       uint32_t K, uint32_t n_groups, Coefs cf, float lr) {
  extern __shared__ float tab[];  // n_groups x 256
  const uint32_t g_first = k_base / 8;
  // Table entry (g, b): sum over the group's 8 probe slots of +-c (bit set: +c), slots
  // outside [k_base, k_base + K) contributing 0; summed pairwise.
  for (uint32_t e = threadIdx.x; e < n_groups * 256u; e += kBlock) {
    const uint32_t g = e >> 8, b = e & 255u;
    float v[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint32_t k = 8u * (g_first + g) + s;
      float cv = 0.0f;
      if (k >= k_base && k - k_base < K) cv = cf.c[k - k_base];
      v[s] = ((b >> s) & 1u) ? cv : -cv;
    }
    tab[e] = ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
  }
  __syncthreads();

  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; i < sp.n_tiles; i += stride) {
    const uint64_t t = sp.t_first + i;
    float acc[kTile];
    if constexpr (NG > 0) {
      group_tree<0, NG, false>(acc, tab, t, step, g_first, 0, NG, k0, k1);
    } else {
      float comp[kTile];
#pragma unroll
      for (int j = 0; j < (int)kTile; ++j) acc[j] = comp[j] = 0.0f;
      for (uint32_t gc = 0; gc < n_groups; gc += 8) {
        float part[kTile];
        group_tree<0, 8, true>(part, tab, t, step, g_first, gc, n_groups, k0, k1);
        // Kahan-Babuska (Neumaier) compensated accumulation across chunks.
#pragma unroll
        for (int j = 0; j < (int)kTile; ++j) {
          const float s = acc[j] + part[j];
          comp[j] += (fabsf(acc[j]) >= fabsf(part[j])) ? ((acc[j] - s) + part[j]) : ((part[j] - s) + acc[j]);
          acc[j] = s;
        }
      }
#pragma unroll
      for (int j = 0; j < (int)kTile; ++j) acc[j] = acc[j] + comp[j];
    }
    apply_tile<S, VEC>(params, sp, t, [&](int j, float v) { return v - lr * acc[j]; });
  }
}

// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void gen_bits_kernel(uint8_t* out, uint64_t tile_begin, uint64_t n_tiles,
                                                         uint32_t step, uint32_t group, uint32_t k0,
                                                         uint32_t k1) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n_tiles; i += stride) {
    const uint4 r = tile_block(tile_begin + i, step, group, k0, k1);
    const u32x4 w = {r.x, r.y, r.z, r.w};
    *reinterpret_cast<u32x4*>(out + 16 * i) = w;
  }
}

// ---------------------------------------------------------------------------------------
// Host side.
uint32_t grid_for(uint64_t n_tiles) {
  const uint64_t cap = g_max_blocks ? g_max_blocks : kDefaultMaxBlocks;
  const uint64_t need = (n_tiles + kBlock - 1) / kBlock;
  return static_cast<uint32_t>(need < cap ? need : cap);
}

int check_params(const void* params, zo_dtype dt, uint64_t offset, uint64_t n, size_t* elem) {
  if (dt != ZO_F32 && dt != ZO_BF16) return ZO_ERR_ARG;
  *elem = dt == ZO_F32 ? 4 : 2;
  if (n == 0) return ZO_OK;
  if (params == nullptr) return ZO_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(params) % *elem != 0) return ZO_ERR_ARG;
  if (offset + n < offset) return ZO_ERR_ARG;  // wraps past 2^64
  return ZO_OK;
}

Span make_span(uint64_t offset, uint64_t n) {
  Span sp;
  sp.lo = offset;
  sp.hi = offset + n;
  sp.t_first = offset / kTile;
  sp.n_tiles = (sp.hi - 1) / kTile - sp.t_first + 1;
  return sp;
}

// Full tiles can move as 16-byte vectors iff the address of global element 0 (params
// shifted back by offset elements) is 16-byte aligned, since tiles span 32 or 64 bytes.
bool vector_ok(const void* params, uint64_t offset, size_t elem) {
  const uintptr_t base = reinterpret_cast<uintptr_t>(params) - static_cast<uintptr_t>(offset * elem);
  return (base & 15u) == 0;
}

int launch_status() { return hipGetLastError() == hipSuccess ? ZO_OK : ZO_ERR_HIP; }

template <class S, bool VEC>
void launch_update(void* params, const Span& sp, uint32_t k0, uint32_t k1, uint32_t step, uint32_t k_base,
                   uint32_t K, uint32_t n_groups, const Coefs& cf, float lr, hipStream_t st) {
  const dim3 grid(grid_for(sp.n_tiles)), block(kBlock);
  const size_t lds = static_cast<size_t>(n_groups) * 256 * sizeof(float);
  auto* p = static_cast<typename S::storage*>(params);
  switch (n_groups) {
    case 1: update_kernel<S, VEC, 1><<<grid, block, lds, st>>>(p, sp, k0, k1, step, k_base, K, n_groups, cf, lr); break;
    case 2: update_kernel<S, VEC, 2><<<grid, block, lds, st>>>(p, sp, k0, k1, step, k_base, K, n_groups, cf, lr); break;
    case 4: update_kernel<S, VEC, 4><<<grid, block, lds, st>>>(p, sp, k0, k1, step, k_base, K, n_groups, cf, lr); break;
    case 8: update_kernel<S, VEC, 8><<<grid, block, lds, st>>>(p, sp, k0, k1, step, k_base, K, n_groups, cf, lr); break;
    default: update_kernel<S, VEC, 0><<<grid, block, lds, st>>>(p, sp, k0, k1, step, k_base, K, n_groups, cf, lr); break;
  }
}

template <class S, bool VEC>
void launch_perturb(void* params, const Span& sp, uint32_t k0, uint32_t k1, uint32_t step, uint32_t k,
                    float eps, hipStream_t st) {
  perturb_kernel<S, VEC><<<dim3(grid_for(sp.n_tiles)), dim3(kBlock), 0, st>>>(
      static_cast<typename S::storage*>(params), sp, k0, k1, step, k / 8, k % 8, eps);
}

}  // namespace

extern "C" {

int zo_perturb(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
               uint32_t k, float eps, void* stream) {
  size_t elem = 0;
  const int rc = check_params(params, dtype, offset, n, &elem);
  if (rc != ZO_OK) return rc;
  if (!std::isfinite(eps)) return ZO_ERR_NONFINITE;
  if (n == 0) return ZO_OK;
  const Span sp = make_span(offset, n);
  const uint32_t k0 = static_cast<uint32_t>(seed), k1 = static_cast<uint32_t>(seed >> 32);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool vec = vector_ok(params, offset, elem);
  (void)hipGetLastError();
  if (dtype == ZO_F32) {
    vec ? launch_perturb<F32, true>(params, sp, k0, k1, step, k, eps, st)
        : launch_perturb<F32, false>(params, sp, k0, k1, step, k, eps, st);
  } else {
    vec ? launch_perturb<BF16, true>(params, sp, k0, k1, step, k, eps, st)
        : launch_perturb<BF16, false>(params, sp, k0, k1, step, k, eps, st);
  }
  return launch_status();
}

int zo_update_ex(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
                 uint32_t k_base, uint32_t K, const float* c, float lr, void* stream) {
  size_t elem = 0;
  const int rc = check_params(params, dtype, offset, n, &elem);
  if (rc != ZO_OK) return rc;
  if (K > ZO_K_MAX) return ZO_ERR_ARG;
  if (static_cast<uint64_t>(k_base) + K > (1ull << 32)) return ZO_ERR_ARG;
  if (K > 0 && c == nullptr) return ZO_ERR_NULL;
  if (!std::isfinite(lr)) return ZO_ERR_NONFINITE;
  for (uint32_t j = 0; j < K; ++j)
    if (!std::isfinite(c[j])) return ZO_ERR_NONFINITE;
  if (n == 0 || K == 0) return ZO_OK;
  Coefs cf;
  for (uint32_t j = 0; j < ZO_K_MAX; ++j) cf.c[j] = j < K ? c[j] : 0.0f;
  const uint32_t g_first = k_base / 8;
  const uint32_t g_last = static_cast<uint32_t>((static_cast<uint64_t>(k_base) + K - 1) / 8);
  const uint32_t n_groups = g_last - g_first + 1;
  const Span sp = make_span(offset, n);
  const uint32_t k0 = static_cast<uint32_t>(seed), k1 = static_cast<uint32_t>(seed >> 32);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool vec = vector_ok(params, offset, elem);
  (void)hipGetLastError();
  if (dtype == ZO_F32) {
    vec ? launch_update<F32, true>(params, sp, k0, k1, step, k_base, K, n_groups, cf, lr, st)
        : launch_update<F32, false>(params, sp, k0, k1, step, k_base, K, n_groups, cf, lr, st);
  } else {
    vec ? launch_update<BF16, true>(params, sp, k0, k1, step, k_base, K, n_groups, cf, lr, st)
        : launch_update<BF16, false>(params, sp, k0, k1, step, k_base, K, n_groups, cf, lr, st);
  }
  return launch_status();
}

int zo_update(void* params, zo_dtype dtype, uint64_t n, uint64_t seed, uint32_t step, uint32_t K,
              const float* c, float lr, void* stream) {
  return zo_update_ex(params, dtype, 0, n, seed, step, 0, K, c, lr, stream);
}

int zo_gen_bits(uint8_t* out_dev, uint64_t tile_begin, uint64_t n_tiles, uint64_t seed, uint32_t step,
                uint32_t group, void* stream) {
  if (n_tiles == 0) return ZO_OK;
  if (out_dev == nullptr) return ZO_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(out_dev) % 16 != 0) return ZO_ERR_ARG;
  if (tile_begin >= (1ull << 60) || n_tiles > (1ull << 60) - tile_begin) return ZO_ERR_ARG;
  (void)hipGetLastError();
  gen_bits_kernel<<<dim3(grid_for(n_tiles)), dim3(kBlock), 0, static_cast<hipStream_t>(stream)>>>(
      out_dev, tile_begin, n_tiles, step, group, static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
  return launch_status();
}

void zo_set_max_blocks(uint32_t max_blocks) { g_max_blocks = max_blocks; }

}  // extern "C"
