// Probe regenerate-and-apply sweeps of 1.5-SPSA for gfx950 (CDNA4).
//
// zo_perturb applies theta + eps z_k (Algorithm 1's +eps / -2 eps / +eps applications),
// zo_update applies theta - lr sum_k c_k z_k in one pass (section 4.2, Eq. 6), and
// zo_gen_bits exposes the probe generator. Probes are regenerated in registers from
// (seed, step, k, element index) with Philox4x32-10 (Salmon et al., SC'11): one 128-bit
// block per 16-element tile and probe group of 8, 8 probe signs per byte (section 4.3).
// Nothing but theta touches HBM.
//
// Each lane runs one Philox block per row group (1024 elements, zo_stream.h) and probe group:
// bf16 lane pairs then swap two generator words (v_permlane32_swap, two instructions) and
// fp32 lane groups transpose a 4x4 word matrix (v_permlane32_swap / v_permlane16_swap, four
// instructions), so that every lane holds the probe bytes of its own vectors. Large sweeps cap
// the workgroups per CU (few long read-write streams keep HBM busiest), and the lightest
// perturbs are paced.
//
// zo_perturb_segments / zo_update_segments sweep a list of separate tensors: the host validates
// the list, builds one plan per tensor and launches batches of up to 64 plans (kernel
// arguments); inside a launch the chunk slots and edge tiles of all its tensors are numbered
// consecutively (slots aligned to memory, zo_plan.h) and each wave finds its chunk's tensor
// by a binary search.
//
// The update keeps, per probe group, a 256-entry table in LDS: entry b is lr times the signed
// sum of the group's 8 coefficients selected by the bits of b (pairwise), so applying 8 probes
// to an element costs a byte extract and an LDS read, and the step is one subtraction. The
// restore of a probe in one of the update's groups is merged into that group's entries. In
// streaming launches the tables are spread over 16 or 32 copies so that lanes read different
// LDS banks. Groups accumulate in fp32, sequentially within runs of 8 groups and with Neumaier
// compensation across runs.
//
// Built with -ffp-contract=off: every product and sum is rounded as written.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <type_traits>

#include "zo.h"
#include "zo_plan.h"
#include "zo_stream.h"

namespace {

using namespace zo;

constexpr int kRounds = 10;

// ---------------------------------------------------------------------------------------
// Philox4x32-R: round (x0,x1,x2,x3) -> (hi(M1 x2)^x1^k0, lo(M1 x2), hi(M0 x0)^x3^k1, lo(M0 x0)),
// key bumped by the Weyl constants after each round. 32x32->64 products: v_mad_u64_u32; each
// three-way XOR is one v_bitop3_b32 (truth table 0x96), which the compiler does not form from
// a ^ b ^ c by itself.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox4x32(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                            uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * x0;
    const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * x2;
    const uint32_t y0 = xor3(static_cast<uint32_t>(p1 >> 32), x1, k0);
    const uint32_t y2 = xor3(static_cast<uint32_t>(p0 >> 32), x3, k1);
    x1 = static_cast<uint32_t>(p1);
    x3 = static_cast<uint32_t>(p0);
    x0 = y0;
    x2 = y2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(x0, x1, x2, x3);
}

// The block of tile t and probe group `group`: counter (t mod 2^32, t / 2^32, step, group).
__device__ __forceinline__ uint4 gen_block(const Gen& gen, uint64_t t, uint32_t group) {
  return philox4x32(static_cast<uint32_t>(t), static_cast<uint32_t>(t >> 32), gen.step, group, gen.k0, gen.k1);
}

// Byte e (0..3) of a generator word: the probe byte of one element.
__device__ __forceinline__ uint32_t word_byte(uint32_t w, int e) { return (w >> (8 * e)) & 0xFFu; }

// Table entry selected by byte e of w, in a table of 256 floats. The byte offset is one SDWA
// shift for every byte (the compiler turns byte 0 into a shift and a mask unless told).
__device__ __forceinline__ float table_at(const float* tab, uint32_t w, int e) {
  uint32_t off;
  if (e == 0)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
        : "=v"(off)
        : "v"(w));
  else
    off = ((w >> (8 * e)) & 0xFFu) << 2;
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(tab) + off);
}

// For a row group starting at global vector vbase (a multiple of GroupShape::kVecs) and probe
// group g: W[u][w] = the generator words this lane's vector in row u needs.
// bf16: lanes m and m + 32 hold the two halves of tile T(u) = vbase/2 + 32u + m; lane m + 32q
// generates tile T(q), and one permlane32 swap per word pair hands each lane the half it
// needs (x,y for the first half, z,w for the second).
__device__ __forceinline__ void group_words(const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t group,
                                            uint32_t (&W)[2][BF16::kWords], BF16) {
  const uint32_t q = lane >> 5, m = lane & 31u;
  const uint4 r = gen_block(gen, vbase / 2 + 32ull * q + m, group);
  const auto sx = __builtin_amdgcn_permlane32_swap(r.x, r.z, false, false);
  const auto sy = __builtin_amdgcn_permlane32_swap(r.y, r.w, false, false);
  W[0][0] = sx[0];
  W[0][1] = sy[0];
  W[1][0] = sx[1];
  W[1][1] = sy[1];
}

// fp32: lanes m + 16q (q = 0..3) hold the four quarters of tile T(u) = vbase/4 + 16u + m;
// lane m + 16q generates tile T(q), and a 4x4 transpose across the four lanes (permlane32
// swaps exchange the off-diagonal 2x2 blocks, permlane16 swaps the elements inside them)
// leaves word q of tile T(u) in register u.
__device__ __forceinline__ void group_words(const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t group,
                                            uint32_t (&W)[4][F32::kWords], F32) {
  const uint32_t q = lane >> 4, m = lane & 15u;
  const uint4 r = gen_block(gen, vbase / 4 + 16ull * q + m, group);
  uint32_t a[4] = {r.x, r.y, r.z, r.w};
  auto sw32 = [&](int i, int j) {
    const auto p = __builtin_amdgcn_permlane32_swap(a[i], a[j], false, false);
    a[i] = p[0];
    a[j] = p[1];
  };
  auto sw16 = [&](int i, int j) {
    const auto p = __builtin_amdgcn_permlane16_swap(a[i], a[j], false, false);
    a[i] = p[0];
    a[j] = p[1];
  };
  sw32(0, 2);
  sw32(1, 3);
  sw16(0, 1);
  sw16(2, 3);
#pragma unroll
  for (int u = 0; u < 4; ++u) W[u][0] = a[u];
}

// Probe byte of element e (0 .. kVecElems-1) of a vector, from its words.
template <class S>
__device__ __forceinline__ uint32_t elem_byte(const uint32_t (&w)[S::kWords], int e) {
  return word_byte(w[e >> 2], e & 3);
}

// ---------------------------------------------------------------------------------------
// perturb: theta + eps * z_k (bit k mod 8 of each probe byte of group k / 8). TWO: the
// fused transition theta + (eps_a z_a + eps_b z_b), the pair's sum rounded to fp32 first.
__device__ __forceinline__ float delta(const Probe& p, uint32_t byte) { return ((byte >> p.bit) & 1u) ? p.eps : -p.eps; }

template <class S, bool TWO, int N, int PACE, int BLOCK, int WPS>
__global__ __launch_bounds__(BLOCK) void perturb_kernel(Plans<N> ps, Gen gen, Probe a, Probe b) {
  extern __shared__ uint32_t occupancy_pad[];  // dynamic LDS only limits workgroups per CU
  if (ps.count == 0xFFFFFFFFu) occupancy_pad[threadIdx.x] = 0;  // never taken (count <= 64)
  constexpr int R = GroupShape<S>::kRows;
  const bool shared_group = a.group == b.group;
  auto no_prologue = []() {};
  for_each_group<S, 2, N, PACE, BLOCK, WPS>(ps, [&](uint64_t vbase, u32x4 (&d)[R], uint32_t lane) {
    uint32_t Wa[R][S::kWords], Wb[R][S::kWords];
    group_words(gen, vbase, lane, a.group, Wa, S());
    if (TWO) {
      if (shared_group) {
#pragma unroll
        for (int u = 0; u < R; ++u)
#pragma unroll
          for (int q = 0; q < S::kWords; ++q) Wb[u][q] = Wa[u][q];
      } else {
        group_words(gen, vbase, lane, b.group, Wb, S());
      }
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float v[S::kVecElems];
      S::unpack(d[u], v);
#pragma unroll
      for (int e = 0; e < S::kVecElems; ++e) {
        float dv = delta(a, elem_byte<S>(Wa[u], e));
        if (TWO) dv = dv + delta(b, elem_byte<S>(Wb[u], e));
        v[e] = v[e] + dv;
      }
      d[u] = S::pack(v);
    }
  }, no_prologue);
  for_each_edge<N, BLOCK>(ps, [&](const Plan& pl, uint64_t t) {
    const uint4 ra = gen_block(gen, t, a.group);
    const uint4 rb = TWO ? gen_block(gen, t, b.group) : ra;
    const uint32_t xa[4] = {ra.x, ra.y, ra.z, ra.w}, xb[4] = {rb.x, rb.y, rb.z, rb.w};
    tile_elementwise<S>(reinterpret_cast<typename S::storage*>(pl.base), pl.lo, pl.hi, t, [&](int e, float v) {
      float dv = delta(a, word_byte(xa[e >> 2], e & 3));
      if (TWO) dv = dv + delta(b, word_byte(xb[e >> 2], e & 3));
      return v + dv;
    });
  });
}

// ---------------------------------------------------------------------------------------
// update: theta - lr * sum_k c_k z_k.

// Spread tables, for streaming launches: C = 32 or 16 copies of each 256-entry table,
// interleaved in planes of 64 KiB that hold P = 64 / C groups each (at most two planes): copy
// r of entry e of group g is float 16384 (g / P) + 64 e + C (g mod P) + r. Lane l reads copy
// l mod C, which sits in LDS bank (C (g mod P) + l mod C) mod 32: with 32 copies every lane of
// a half-wave has its own bank, so a 64-lane read of random bytes takes 2 LDS cycles instead
// of about 6.3 when all lanes share one copy; with 16 copies two lanes share a bank, about 4
// cycles. A lookup's byte address, 65536 (g / P) + 256 e + 4 (l mod C) + 4 C (g mod P), is one
// byte permute of the generator word and the lane's offset word (byte 0: 4 (l mod C), byte 2:
// 1, selected for the second plane), plus an immediate offset: as many instructions as a
// lookup into a shared table.
constexpr uint32_t kSpreadFloats = 256 * 64;  // one plane
template <int C>
constexpr uint32_t groups_per_plane() {
  return C > 0 ? 64 / C : 1;
}
// floats of the tables of NG groups: C interleaved copies, or one shared copy (C = 0)
template <int NG, int C>
constexpr uint32_t table_floats() {
  static_assert(C == 0 || ((C == 16 || C == 32) && NG * C <= 128), "spread tables fill at most two planes");
  return C == 0 ? NG * 256 : (NG * C <= 64 ? 1 : 2) * kSpreadFloats;
}

// Build the n_groups x 256 table in LDS (C > 0: the interleaved copies). Entry (g, b):
// fl(lr * t), t the sum over the group's 8 probe slots of +-c (bit set: +c), pairwise; slots
// outside [k_base, k_base + K) contribute 0. Scaling each entry once here saves the sweep a
// multiply per element; with one probe the entry is +-fl(lr * c), the step a perturb by
// -fl(lr * c) would apply. A restore probe in group fold_g (the update's own probe groups hold
// the probe Algorithm 1 restores last) is merged into that group's entries: fl(fl(lr * t) -
// delta), delta = +-eps_r by the probe's bit of b, so the sweep applies theta + delta - sum
// with no per-element work of its own. Thread b writes entry b of every group: the group loop
// and the coefficient reads are uniform (scalar loads), and the sign of slot s is an XOR of the
// coefficient's sign bit with bit s of ~b. A workgroup of BLOCK threads builds BLOCK / 256
// groups at a time: thread b + 256 m writes entry b of groups m, m + BLOCK / 256, ...
template <int C, int BLOCK>
__device__ __forceinline__ void build_tables(float* tab, const Coefs& cf, uint32_t k_base, uint32_t K,
                                             uint32_t n_groups, float lr, uint32_t fold_g, const Probe& fold) {
  static_assert(BLOCK % 256 == 0, "one table entry per thread");
  const uint32_t b = threadIdx.x & 255u;
  uint32_t flip[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) flip[s] = ((~b) << (31 - s)) & 0x80000000u;
  const uint32_t g_first = k_base / 8;
  for (uint32_t g = threadIdx.x >> 8; g < n_groups; g += BLOCK / 256) {
    float v[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint32_t k = 8u * (g_first + g) + s;
      const float cv = (k >= k_base && k - k_base < K) ? cf.c[k - k_base] : 0.0f;
      v[s] = __uint_as_float(__float_as_uint(cv) ^ flip[s]);
    }
    float t = (((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]))) * lr;
    if (g == fold_g) t = t - delta(fold, b);
    if constexpr (C > 0) {
      // entry b's C / 4 float4 of copies, 256 bytes after entry b - 1's: thread b writes them
      // starting at float4 b mod (C / 4), so that the lanes of each write spread over the banks
      // the group's copies occupy (in a fixed order all 64 would land on the same 4 banks)
      constexpr uint32_t Q = C / 4, P = groups_per_plane<C>();
      float* e = tab + kSpreadFloats * (g / P) + 64u * b + C * (g % P);
      const float4 t4 = make_float4(t, t, t, t);
#pragma unroll
      for (uint32_t q = 0; q < Q; ++q) *reinterpret_cast<float4*>(e + 4u * ((q + b) & (Q - 1))) = t4;
    } else {
      tab[256u * g + b] = t;
    }
  }
  __syncthreads();
}

// Spread-table lookup in group g (C copies): one byte permute forms the address (byte 0: the
// lane's copy offset, byte 0 of `lane_off` = 4 (l mod C); byte 1: byte e of w; byte 2: 0, or
// for the second plane byte 2 of lane_off, which is 1; byte 3: 0), then the float there plus
// the group's offset 4 C (g mod P) inside its plane.
template <int C>
__device__ __forceinline__ float spread_at(const float* tab, uint32_t lane_off, uint32_t w, int e, uint32_t g) {
  constexpr uint32_t P = groups_per_plane<C>();
  const uint32_t plane_sel = g / P ? 0x00020000u : 0x000C0000u;
  const uint32_t addr =
      __builtin_amdgcn_perm(w, lane_off, 0x0C000000u | plane_sel | ((4u + static_cast<uint32_t>(e)) << 8));
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(tab) + addr + 4u * C * (g % P));
}

// acc[u][e] (+)= table value of probe group g for each element of the row group; W receives
// the group's generator words.
template <class S, bool FIRST, int C>
__device__ __forceinline__ void add_group(float (&acc)[GroupShape<S>::kRows][S::kVecElems], const float* tab,
                                          const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t g,
                                          uint32_t g_first, uint32_t lane_off,
                                          uint32_t (&W)[GroupShape<S>::kRows][S::kWords]) {
  constexpr int R = GroupShape<S>::kRows;
  group_words(gen, vbase, lane, g_first + g, W, S());
  const float* tg = tab + 256u * g;
#pragma unroll
  for (int u = 0; u < R; ++u)
#pragma unroll
    for (int e = 0; e < S::kVecElems; ++e) {
      float x;
      if constexpr (C > 0)
        x = spread_at<C>(tab, lane_off, W[u][e >> 2], e & 3, g);
      else
        x = table_at(tg, W[u][e >> 2], e & 3);
      acc[u][e] = FIRST ? x : acc[u][e] + x;
    }
}

// Sum of the tables of probe groups 0 .. n_groups-1 for the row group: NG > 0 fixes the count
// at compile time (one run); NG == 0: runs of 8 groups, Neumaier-compensated across runs.
template <class S, int NG, int C>
__device__ __forceinline__ void group_sums(float (&acc)[GroupShape<S>::kRows][S::kVecElems], const float* tab,
                                           const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t n_groups,
                                           uint32_t g_first, uint32_t lane_off) {
  constexpr int R = GroupShape<S>::kRows;
  static_assert(C == 0 || NG > 0, "spread tables need a fixed group count");
  uint32_t W[R][S::kWords];
  if constexpr (NG > 0) {
    add_group<S, true, C>(acc, tab, gen, vbase, lane, 0, g_first, lane_off, W);
#pragma unroll
    for (int g = 1; g < NG; ++g)
      add_group<S, false, C>(acc, tab, gen, vbase, lane, g, g_first, lane_off, W);
  } else {
    float comp[R][S::kVecElems];
    for (uint32_t g0 = 0; g0 < n_groups; g0 += 8) {
      float part[R][S::kVecElems];
      add_group<S, true, 0>(part, tab, gen, vbase, lane, g0, g_first, lane_off, W);
      const uint32_t g1 = n_groups - g0 < 8 ? n_groups : g0 + 8;
      for (uint32_t g = g0 + 1; g < g1; ++g)
        add_group<S, false, 0>(part, tab, gen, vbase, lane, g, g_first, lane_off, W);
#pragma unroll
      for (int u = 0; u < R; ++u)
#pragma unroll
        for (int e = 0; e < S::kVecElems; ++e) {
          if (g0 == 0) {
            acc[u][e] = part[u][e];
            comp[u][e] = 0.0f;
          } else {
            const float a = acc[u][e], p = part[u][e], s = a + p;
            comp[u][e] += fabsf(a) >= fabsf(p) ? (a - s) + p : (p - s) + a;
            acc[u][e] = s;
          }
        }
    }
#pragma unroll
    for (int u = 0; u < R; ++u)
#pragma unroll
      for (int e = 0; e < S::kVecElems; ++e) acc[u][e] = acc[u][e] + comp[u][e];
  }
}

// Same sum for one tile on the element-wise path (one lane, all 16 elements).
template <int C>
__device__ __forceinline__ void tile_sums(float (&acc)[kTile], const float* tab, const Gen& gen, uint64_t t,
                                          uint32_t n_groups, uint32_t g_first) {
  float comp[kTile];
  for (uint32_t g0 = 0; g0 < n_groups; g0 += 8) {
    float part[kTile];
    const uint32_t g1 = n_groups - g0 < 8 ? n_groups : g0 + 8;
    for (uint32_t g = g0; g < g1; ++g) {
      const uint4 r = gen_block(gen, t, g_first + g);
      const uint32_t x[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int j = 0; j < (int)kTile; ++j) {
        const uint32_t byte = word_byte(x[j >> 2], j & 3);
        float v;
        if constexpr (C > 0) {
          constexpr uint32_t P = groups_per_plane<C>();
          v = tab[kSpreadFloats * (g / P) + 64u * byte + C * (g % P) + (threadIdx.x % C)];
        } else {
          v = tab[256u * g + byte];
        }
        part[j] = g == g0 ? v : part[j] + v;
      }
    }
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) {
      if (g0 == 0) {
        acc[j] = part[j];
        comp[j] = 0.0f;
      } else {
        const float a = acc[j], p = part[j], s = a + p;
        comp[j] += fabsf(a) >= fabsf(p) ? (a - s) + p : (p - s) + a;
        acc[j] = s;
      }
    }
  }
  if (n_groups > 8) {
#pragma unroll
    for (int j = 0; j < (int)kTile; ++j) acc[j] = acc[j] + comp[j];
  }
}

// How an update applies a restore probe r (theta + eps_r z_r - lr * sum, the restore merged
// with the update): kNoRestore, none; kFolded, r lies in one of the update's probe groups and
// is folded into that group's table (see build_tables), so the per-element work is the plain
// update's; kPerElement, r lies outside them and is applied per element as t =
// fl(theta + delta_r), then t minus the sum of the table values, its generator words made
// after the group loop.
enum RestoreMode { kNoRestore = 0, kFolded = 1, kPerElement = 2 };

template <class S, int NG, int RESTORE, int N, int C, int BLOCK, int WPS, int PACE = 0, int AHEAD = 0>
__global__ __launch_bounds__(BLOCK) void update_kernel(Plans<N> ps, Gen gen, uint32_t k_base, uint32_t K,
                                                      uint32_t n_groups, Coefs cf, float lr, Probe r) {
  // n_groups x 256 floats (C > 0: the interleaved copies): static for a fixed group count
  // (constant LDS offsets), else dynamic.
  extern __shared__ float tab_dyn[];
  __shared__ float tab_fix[NG > 0 ? table_floats<NG, C>() : 1];
  float* tab = NG > 0 ? tab_fix : tab_dyn;
  const uint32_t g_first = k_base / 8;
  // the table a folded restore changes (none: a group index no table has; below g_first wraps)
  const uint32_t fold_g = RESTORE == kFolded ? r.group - g_first : 0xFFFFFFFFu;
  // the tables are built while each wave's first loads are in flight (for_each_group's prologue)
  auto build = [&]() { build_tables<C, BLOCK>(tab, cf, k_base, K, n_groups, lr, fold_g, r); };
  // the lane's copy of a spread table (byte 0) and the second plane's offset (byte 2)
  const uint32_t lane_off = 4u * (threadIdx.x % (C > 0 ? C : 32)) | (1u << 16);
  constexpr int R = GroupShape<S>::kRows;
  // two groups in flight with spread tables and for one, two or four groups; one for the
  // other counts, which run at three or more workgroups per CU (AHEAD > 0 sets it)
  constexpr int kAhead = AHEAD ? AHEAD : C > 0 || NG == 1 || NG == 2 || NG == 4 ? 2 : 1;
  for_each_group<S, kAhead, N, PACE, BLOCK, WPS>(ps, [&](uint64_t vbase, u32x4 (&d)[R], uint32_t lane) {
    float acc[R][S::kVecElems];
    uint32_t Wr[R][S::kWords];  // the restore probe's words
    group_sums<S, NG, C>(acc, tab, gen, vbase, lane, n_groups, g_first, lane_off);
    if (RESTORE == kPerElement) group_words(gen, vbase, lane, r.group, Wr, S());
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float v[S::kVecElems];
      S::unpack(d[u], v);
#pragma unroll
      for (int e = 0; e < S::kVecElems; ++e) {
        if (RESTORE == kPerElement) v[e] = v[e] + delta(r, elem_byte<S>(Wr[u], e));
        v[e] = v[e] - acc[u][e];
      }
      d[u] = S::pack(v);
    }
  }, build);
  for_each_edge<N, BLOCK>(ps, [&](const Plan& pl, uint64_t t) {
    float acc[kTile];
    tile_sums<C>(acc, tab, gen, t, n_groups, g_first);
    const uint4 rr = RESTORE == kPerElement ? gen_block(gen, t, r.group) : make_uint4(0, 0, 0, 0);
    const uint32_t xr[4] = {rr.x, rr.y, rr.z, rr.w};
    tile_elementwise<S>(reinterpret_cast<typename S::storage*>(pl.base), pl.lo, pl.hi, t, [&](int e, float v) {
      if (RESTORE == kPerElement) v = v + delta(r, word_byte(xr[e >> 2], e & 3));
      return v - acc[e];
    });
  });
}

// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void gen_bits_kernel(uint8_t* out, uint64_t tile_begin, uint64_t n_tiles,
                                                         uint32_t group, Gen gen) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n_tiles; i += stride) {
    const uint4 r = gen_block(gen, tile_begin + i, group);
    *reinterpret_cast<u32x4*>(out + 16 * i) = u32x4{r.x, r.y, r.z, r.w};
  }
}

// ---------------------------------------------------------------------------------------
// Host side.
int launch_status() { return hipGetLastError() == hipSuccess ? ZO_OK : ZO_ERR_HIP; }

// A workgroup's LDS above 64 KiB (static plus dynamic) must be allowed per kernel before the
// launch.
template <class K>
void allow_lds(K kernel, size_t dynamic_bytes, size_t static_bytes = 0) {
  if (dynamic_bytes + static_bytes > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(dynamic_bytes));
}

// Launch dimensions a kernel is built for: workgroup size and waves per stream. A kernel is
// always launched with the dimensions it was built for.
template <int B, int W>
struct Dims {
  static constexpr int block = B, wps = W;
};

template <class S, int N>
void launch_sweep(const Plans<N>& ps, const Gen& gen, const Sweep& w, const Shape& sh, hipStream_t st) {
  const uint32_t cap = sh.blocks_per_cu;
  // the grid of a launch with B threads per workgroup and W waves per stream
  auto grid_of = [&](uint32_t B, uint32_t W) {
    Shape s = sh;
    s.block = B;
    s.wps = W;
    return dim3(plans_grid(ps, s));
  };
  if (!w.update) {
    const size_t pad = occupancy_lds(cap, 0);
    auto go = [&](auto kernel, Probe b) {
      allow_lds(kernel, pad);
      kernel<<<grid_of(kBlock, 1), dim3(kBlock), pad, st>>>(ps, gen, w.a, b);
    };
    // paced when the generator work per byte is lightest: one probe group, or fp32 with two;
    // at 4 outstanding operations (bf16: one probe +1.3%, two in one group +3.4% over 2; fp32
    // one probe +3%), the fp32 two-probe perturb at 2 (4 measured equal or lower)
    constexpr int kPace2 = sizeof(typename S::storage) == 2 ? 4 : 2;
    const bool two_groups = w.two && w.a.group != w.b.group;
    const bool paced = (two_groups ? 2u : 1u) * (sizeof(typename S::storage) == 2 ? 2u : 1u) <= 2u;
    if (w.two)
      paced ? go(perturb_kernel<S, true, N, kPace2, kBlock, 1>, w.b) : go(perturb_kernel<S, true, N, 0, kBlock, 1>, w.b);
    else
      paced ? go(perturb_kernel<S, false, N, 4, kBlock, 1>, w.a) : go(perturb_kernel<S, false, N, 0, kBlock, 1>, w.a);
    return;
  }
  const uint32_t copies = sh.copies;
  // One kernel: NG groups fixed at compile time (0: a runtime count, tables in dynamic LDS), C
  // copies of each table, launched with the dimensions it was built for.
  auto go = [&](auto kernel, auto groups, auto copies_c, auto dims) {
    constexpr int NG = decltype(groups)::value, C = decltype(copies_c)::value;
    constexpr int B = decltype(dims)::block, W = decltype(dims)::wps;
    const size_t table_bytes = NG > 0 ? size_t{table_floats<NG, C>()} * sizeof(float)
                                      : static_cast<size_t>(w.n_groups) * 256 * sizeof(float);
    const size_t static_lds = NG > 0 ? table_bytes : 0;
    const size_t pad = occupancy_lds(cap, static_lds);
    const size_t tables = NG > 0 ? 0 : table_bytes;
    const size_t lds = tables > pad ? tables : pad;  // dynamic tables (up to 128 KiB) or the pad
    allow_lds(kernel, lds, static_lds);
    kernel<<<grid_of(B, W), dim3(B), lds, st>>>(ps, gen, w.k_base, w.K, w.n_groups, w.cf, w.lr, w.r);
  };
  using std::integral_constant;
  using D256 = Dims<kBlock, 1>;
  using C0 = integral_constant<int, 0>;
  // a restore probe outside the update's groups: the per-element restore, runtime group count
  if (w.restore && !w.fold) {
    go(update_kernel<S, 0, kPerElement, N, 0, kBlock, 1>, C0{}, C0{}, D256{});
    return;
  }
  constexpr bool bf16 = sizeof(typename S::storage) == 2;
  using G1 = integral_constant<int, 1>;
  using G2 = integral_constant<int, 2>;
  using G4 = integral_constant<int, 4>;
  using G8 = integral_constant<int, 8>;
  using C16 = integral_constant<int, 16>;
  using C32 = integral_constant<int, 32>;
  // The tables and launch dimensions shape_for picks for each group count: streaming bf16
  // updates of two, four and eight groups take their own (two waves per stream; 1024-thread
  // workgroups); everything else 256 threads. bf16 updates of one and two groups are paced at
  // four outstanding memory operations, as the one-probe perturb. A
  // folded restore runs the same code (its own instantiation, so that profiles tell the two
  // calls apart).
  auto dispatch = [&](auto mode) {
    constexpr int M = decltype(mode)::value;
    switch (w.n_groups) {
      case 1:
        if (copies)
          go(update_kernel<S, 1, M, N, 32, kBlock, 1>, G1{}, C32{}, D256{});
        else
          go(update_kernel<S, 1, M, N, 0, kBlock, 1, bf16 ? 4 : 0>, G1{}, C0{}, D256{});
        break;
      case 2:
        if (!copies)
          go(update_kernel<S, 2, M, N, 0, kBlock, 1>, G2{}, C0{}, D256{});
        else if constexpr (!bf16)
          go(update_kernel<S, 2, M, N, 32, kBlock, 1>, G2{}, C32{}, D256{});
        else
          go(update_kernel<S, 2, M, N, 32, 512, 2, 4>, G2{}, C32{}, Dims<512, 2>{});
        break;
      case 4:
        if constexpr (bf16) {
          if (copies) {
            go(update_kernel<S, 4, M, N, 32, 1024, 1>, G4{}, C32{}, Dims<1024, 1>{});
            break;
          }
        }
        go(update_kernel<S, 4, M, N, 0, kBlock, 1>, G4{}, C0{}, D256{});
        break;
      case 8:
        if constexpr (bf16) {
          if (copies) {
            go(update_kernel<S, 8, M, N, 16, 1024, 1>, G8{}, C16{}, Dims<1024, 1>{});
            break;
          }
        }
        go(update_kernel<S, 8, M, N, 0, kBlock, 1>, G8{}, C0{}, D256{});
        break;
      default:
        go(update_kernel<S, 0, M, N, 0, kBlock, 1>, C0{}, C0{}, D256{});
        break;
    }
  };
  if (w.fold)
    dispatch(integral_constant<int, kFolded>{});
  else
    dispatch(integral_constant<int, kNoRestore>{});
}

// One contiguous tensor.
template <class S>
int run_one(void* params, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step, const Sweep& w, void* stream) {
  const Shape sh = shape_for(n, sizeof(typename S::storage), w);
  const Gen gen = make_gen(seed, step);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const zo_segment seg{params, offset, n};
  (void)hipGetLastError();
  // one launch (several only for a tensor of more than kPieceElems weights without full row groups)
  return plan_segments<1>(&seg, 1, sizeof(typename S::storage), sh.chunk_groups, streams_per_block(sh),
                          [&](const Plans<1>& ps) {
    launch_sweep<S>(ps, gen, w, sh, st);
    return launch_status();
  });
}

int run_one_dt(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
               const Sweep& w, void* stream) {
  const int rc = check_params(params, dtype, offset, n);
  if (rc != ZO_OK) return rc;
  const int rs = check_sweep(w);
  if (rs != ZO_OK) return rs;
  if (n == 0) return ZO_OK;
  return dtype == ZO_F32 ? run_one<F32>(params, offset, n, seed, step, w, stream)
                         : run_one<BF16>(params, offset, n, seed, step, w, stream);
}

// A list of tensors (validated as a whole first), swept in launches of up to kSegsPerLaunch
// segments.
template <class S>
int run_segments(const zo_segment* segs, uint32_t n_segs, uint64_t seed, uint32_t step, const Sweep& w,
                 void* stream) {
  const Gen gen = make_gen(seed, step);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t total = 0;  // the call's weights decide the streaming shape of all its launches
  for (uint32_t i = 0; i < n_segs; ++i) total += segs[i].n;
  Shape sh = shape_for(total, sizeof(typename S::storage), w);
  // at most one chunk per stream: a tensor boundary then idles at most one chunk slot per
  // stream of a workgroup (Qwen3-8B as 399 tensors, K = 60: update 10.4-10.5 -> 9.8-9.9 ms
  // against four chunks per stream)
  if (sh.chunks_per_wave > 1) sh.chunks_per_wave = 1;
  (void)hipGetLastError();
  return plan_segments<kSegsPerLaunch>(segs, n_segs, sizeof(typename S::storage), sh.chunk_groups,
                                       streams_per_block(sh), [&](const Plans<kSegsPerLaunch>& ps) {
                                         launch_sweep<S>(ps, gen, w, sh, st);
                                         return launch_status();
                                       });
}

int run_segments_dt(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype, uint64_t seed, uint32_t step,
                    const Sweep& w, void* stream) {
  const int rc = check_segments(segs, n_segs, dtype);
  if (rc != ZO_OK) return rc;
  const int rs = check_sweep(w);
  if (rs != ZO_OK) return rs;
  return dtype == ZO_F32 ? run_segments<F32>(segs, n_segs, seed, step, w, stream)
                         : run_segments<BF16>(segs, n_segs, seed, step, w, stream);
}

}  // namespace

extern "C" {

int zo_perturb(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
               uint32_t k, float eps, void* stream) {
  return run_one_dt(params, dtype, offset, n, seed, step, perturb_sweep(k, eps, nullptr, 0.0f), stream);
}

int zo_perturb2(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
                uint32_t k_a, float eps_a, uint32_t k_b, float eps_b, void* stream) {
  return run_one_dt(params, dtype, offset, n, seed, step, perturb_sweep(k_a, eps_a, &k_b, eps_b), stream);
}

int zo_update_ex(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
                 uint32_t k_base, uint32_t K, const float* c, float lr, void* stream) {
  const int rc = check_params(params, dtype, offset, n);
  if (rc != ZO_OK) return rc;
  Sweep w;
  const int rs = make_update_sweep(w, k_base, K, c, lr, nullptr);
  if (rs != ZO_OK) return rs;
  if (!w.update || n == 0) return ZO_OK;
  return run_one_dt(params, dtype, offset, n, seed, step, w, stream);
}

int zo_update(void* params, zo_dtype dtype, uint64_t n, uint64_t seed, uint32_t step, uint32_t K,
              const float* c, float lr, void* stream) {
  return zo_update_ex(params, dtype, 0, n, seed, step, 0, K, c, lr, stream);
}

int zo_update_restore(void* params, zo_dtype dtype, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step,
                      uint32_t k_base, uint32_t K, const float* c, float lr, uint32_t k_restore,
                      float eps_restore, void* stream) {
  const int rc = check_params(params, dtype, offset, n);
  if (rc != ZO_OK) return rc;
  const Probe r = make_probe(k_restore, eps_restore);
  Sweep w;
  const int rs = make_update_sweep(w, k_base, K, c, lr, &r);
  if (rs != ZO_OK) return rs;
  if (n == 0 || (!w.update && eps_restore == 0.0f)) return ZO_OK;
  return run_one_dt(params, dtype, offset, n, seed, step, w, stream);
}

int zo_perturb_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype, uint64_t seed, uint32_t step,
                        uint32_t k_a, float eps_a, uint32_t k_b, float eps_b, void* stream) {
  const Sweep w = eps_b == 0.0f ? perturb_sweep(k_a, eps_a, nullptr, 0.0f) : perturb_sweep(k_a, eps_a, &k_b, eps_b);
  return run_segments_dt(segs, n_segs, dtype, seed, step, w, stream);
}

int zo_update_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype, uint64_t seed, uint32_t step,
                       uint32_t k_base, uint32_t K, const float* c, float lr, uint32_t k_restore,
                       float eps_restore, void* stream) {
  const int rc = check_segments(segs, n_segs, dtype);
  if (rc != ZO_OK) return rc;
  const Probe r = make_probe(k_restore, eps_restore);
  Sweep w;
  const int rs = make_update_sweep(w, k_base, K, c, lr, &r);
  if (rs != ZO_OK) return rs;
  if (!w.update && eps_restore == 0.0f) return ZO_OK;
  return run_segments_dt(segs, n_segs, dtype, seed, step, w, stream);
}

int zo_gen_bits(uint8_t* out_dev, uint64_t tile_begin, uint64_t n_tiles, uint64_t seed, uint32_t step,
                uint32_t group, void* stream) {
  if (n_tiles == 0) return ZO_OK;
  if (out_dev == nullptr) return ZO_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(out_dev) % 16 != 0) return ZO_ERR_ARG;
  if (tile_begin >= (1ull << 60) || n_tiles > (1ull << 60) - tile_begin) return ZO_ERR_ARG;
  (void)hipGetLastError();
  gen_bits_kernel<<<dim3(grid_for(n_tiles, kBlock, kBlock)), dim3(kBlock), 0, static_cast<hipStream_t>(stream)>>>(
      out_dev, tile_begin, n_tiles, group, make_gen(seed, step));
  return launch_status();
}

void zo_set_max_blocks(uint32_t max_blocks) { set_max_blocks(max_blocks); }

}  // extern "C"
