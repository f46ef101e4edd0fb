// Probe regenerate-and-apply sweeps of 1.5-SPSA for gfx950 (CDNA4).
//
// zo_perturb applies theta + eps z_k (Algorithm 1's +eps / -2 eps / +eps applications),
// zo_update applies theta - lr sum_k c_k z_k in one pass (section 4.2, Eq. 6), and
// zo_gen_bits exposes the probe generator. Probes are regenerated in registers from
// (seed, step, k, element index) with Philox4x32-10 (Salmon et al., SC'11): one 128-bit
// block per 16-element tile and probe group of 8, 8 probe signs per byte (section 4.3).
// Nothing but theta touches HBM.
//
// Memory layout of a sweep. theta is walked in row groups of 1024 elements: 2 (bf16) or 4
// (fp32) rows of 64 contiguous 16-byte vectors, one vector per lane and row, so each load and
// store instruction of a wave covers 1 KiB of contiguous memory (non-temporal: nothing is
// reused). A tile spans 2 vectors (bf16) or 4 (fp32); the lanes holding one tile are m and
// m + 32 (bf16) or m, m + 16, m + 32, m + 48 (fp32), so that the gfx950 half-wave swaps
// v_permlane32_swap / v_permlane16_swap exchange the generator words: each lane runs one
// Philox block per row group and probe group, then bf16 lane pairs swap two words (two
// instructions) and fp32 lane groups transpose a 4x4 word matrix (four instructions). A wave
// streams a chunk of consecutive row groups (up to 32 KiB) with the loads of the next one or
// two groups in flight while it works on the current one, and large sweeps cap the
// workgroups per CU (few long read-write streams keep HBM busiest). The loops are written so
// that the compiler's memory waits are exact, and the lightest perturbs are paced explicitly.
// Head and tail elements that do not fill a row group (and everything, when the storage is
// not 16-byte aligned relative to the global index) take an element-wise path, one tile per
// lane.
//
// zo_perturb_segments / zo_update_segments sweep a list of separate tensors: the host validates
// the list, builds one plan per tensor and launches batches of up to 64 plans (kernel
// arguments); inside a launch the chunks and edge tiles of all its tensors are numbered
// consecutively and each wave finds its chunk's tensor by a binary search.
//
// The update keeps, per probe group, a 256-entry table in LDS: entry b is lr times the signed
// sum of the group's 8 coefficients selected by the bits of b (pairwise), so applying 8 probes
// to an element costs a byte extract and an LDS read, and the step is one subtraction; with one or two groups in a streaming launch
// the tables are spread over 32 copies so that each lane reads its own LDS bank. Groups
// accumulate in fp32, sequentially within runs of 8 groups and with Neumaier compensation
// across runs.
//
// Built with -ffp-contract=off: every product and sum is rounded as written.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <type_traits>
#include <utility>
#include <vector>

#include "zo.h"

namespace {

constexpr uint32_t kTile = 16;    // elements per generator block
constexpr uint32_t kBlock = 256;  // threads per workgroup (4 waves)
constexpr uint32_t kWavesPerBlock = kBlock / 64;
// s_waitcnt immediate for vmcnt(n), n < 16, that leaves expcnt and lgkmcnt unconstrained
// (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int wait_vmcnt(int n) { return 0x0F70 | n; }
constexpr uint64_t kGroupElems = 1024;      // elements per row group (one Philox block per lane)
constexpr uint64_t kMaxChunkBytes = 32768;  // bytes a wave streams per chunk, at most
constexpr uint32_t kDefaultMaxBlocks = 65536;
constexpr int kRounds = 10;

uint32_t g_max_blocks = 0;  // 0: default

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

struct Gen {
  uint32_t k0, k1, step;
  __device__ __forceinline__ uint4 block(uint64_t t, uint32_t group) const {
    return philox4x32(static_cast<uint32_t>(t), static_cast<uint32_t>(t >> 32), step, group, k0, k1);
  }
};

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

// ---------------------------------------------------------------------------------------
// Storage formats.
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
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// A storage type moves 16-byte vectors of kVecElems elements, widened to fp32. kLanesPerTile
// adjacent lanes hold one 16-element tile; each of them needs kWords of the tile's 4
// generator words (word w carries the probe bytes of tile elements 4w .. 4w+3).
struct F32 {
  typedef float storage;
  static constexpr int kVecElems = 4, kLanesPerTile = 4, kWords = 1;
  __device__ static __forceinline__ void unpack(u32x4 d, float (&v)[kVecElems]) {
    v[0] = __uint_as_float(d.x);
    v[1] = __uint_as_float(d.y);
    v[2] = __uint_as_float(d.z);
    v[3] = __uint_as_float(d.w);
  }
  __device__ static __forceinline__ u32x4 pack(const float (&v)[kVecElems]) {
    return u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
  }
  __device__ static __forceinline__ float load1(const storage* p) { return *p; }
  __device__ static __forceinline__ void store1(storage* p, float v) { *p = v; }
};

struct BF16 {
  typedef uint16_t storage;
  static constexpr int kVecElems = 8, kLanesPerTile = 2, kWords = 2;
  __device__ static __forceinline__ void unpack(u32x4 d, float (&v)[kVecElems]) {
    const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      v[2 * m] = __uint_as_float(w[m] << 16);
      v[2 * m + 1] = __uint_as_float(w[m] & 0xFFFF0000u);
    }
  }
  __device__ static __forceinline__ u32x4 pack(const float (&v)[kVecElems]) {
    return u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                 pack_bf16x2(v[6], v[7])};
  }
  __device__ static __forceinline__ float load1(const storage* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
  __device__ static __forceinline__ void store1(storage* p, float v) {
    *p = static_cast<uint16_t>(pack_bf16x2(v, 0.0f) & 0xFFFFu);
  }
};

// A row group: kRows rows of 64 contiguous 16-byte vectors (one vector per lane and row),
// 1024 elements, i.e. one Philox block per lane and probe group.
template <class S>
struct GroupShape {
  static constexpr int kRows = S::kLanesPerTile;                // bf16 2, fp32 4
  static constexpr uint64_t kVecs = 64ull * kRows;
  static constexpr uint64_t kElems = kVecs * S::kVecElems;
  static constexpr uint64_t kBytes = kVecs * 16;                // bf16 2 KiB, fp32 4 KiB
  static_assert(kElems == kGroupElems, "a row group holds 1024 elements");
};

// Group vector held by a lane (for every row u, lane l holds group vector 64u + vec_of_lane(l)):
// the lanes of one tile sit 32 (bf16) or 16 (fp32) lanes apart.
template <class S>
__device__ __forceinline__ uint32_t vec_of_lane(uint32_t lane) {
  return S::kLanesPerTile == 2 ? 2 * (lane & 31u) + (lane >> 5) : 4 * (lane & 15u) + (lane >> 4);
}

// For a row group starting at global vector vbase (a multiple of GroupShape::kVecs) and probe
// group g: W[u][w] = the generator words this lane's vector in row u needs.
// bf16: lanes m and m + 32 hold the two halves of tile T(u) = vbase/2 + 32u + m; lane m + 32q
// generates tile T(q), and one permlane32 swap per word pair hands each lane the half it
// needs (x,y for the first half, z,w for the second).
__device__ __forceinline__ void group_words(const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t group,
                                            uint32_t (&W)[2][BF16::kWords], BF16) {
  const uint32_t q = lane >> 5, m = lane & 31u;
  const uint4 r = gen.block(vbase / 2 + 32ull * q + m, group);
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
  const uint4 r = gen.block(vbase / 4 + 16ull * q + m, group);
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

// Element-wise path: elements of tile t inside [lo, hi), one lane; params holds global
// element lo.
template <class S, class F>
__device__ __forceinline__ void tile_elementwise(typename S::storage* params, uint64_t lo, uint64_t hi, uint64_t t,
                                                 F f) {
  const uint64_t g0 = t * kTile;
#pragma unroll
  for (int j = 0; j < (int)kTile; ++j) {
    const uint64_t g = g0 + j;
    if (g >= lo && g < hi) {
      typename S::storage* p = params + (g - lo);
      S::store1(p, f(j, S::load1(p)));
    }
  }
}

// One segment: global elements [lo, hi) stored from `base` (the address of global element lo).
// The `span` full row groups from global group g_lo (stored from `gbase`) take the vector
// path, in chunks of up to `chunk_groups` groups aligned to multiples of chunk_groups in the
// global group index: the segment's first chunk starts `head` = g_lo mod chunk_groups groups
// before g_lo. The edge tiles [head_t0, +head_nt) and [tail_t0, +tail_nt) (fewer than 1024
// elements at each end) take the element-wise path. The kernels walk chunks and groups with
// 32-bit indices relative to the segment (compares of 64-bit indices need a vector register
// on gfx950, and writing one that a pending store still reads makes the wave wait for that
// store); the host keeps a segment below 2^30 row groups and a launch below 2^31 chunks.
struct Plan {
  char* base;
  uint64_t lo, hi;
  char* gbase;
  uint64_t g_lo;
  uint32_t head, span;
  uint64_t head_t0, tail_t0;
  uint32_t head_nt, tail_nt;
};

// The segments one launch covers. Their chunks and edge tiles are numbered consecutively:
// segment s owns chunks [chunk_end[s-1], chunk_end[s]) and edge tiles [edge_end[s-1], edge_end[s]).
template <int N>
struct Plans {
  uint32_t count;
  uint32_t chunk_groups;
  uint32_t chunk_end[N];
  uint32_t edge_end[N];
  Plan p[N];
};

// The first segment s in [from, count) with x < ends[s], where ends is nondecreasing and
// x < ends[count - 1]: a binary search, so that finding a chunk's segment costs at most
// log2(N) + 1 argument loads wherever the chunk lies.
template <int N>
__device__ __forceinline__ uint32_t segment_of(const uint32_t (&ends)[N], uint32_t from, uint32_t count, uint32_t x) {
  uint32_t lo = from, hi = count - 1;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (x < ends[mid])
      hi = mid;
    else
      lo = mid + 1;
  }
  return lo;
}

template <class S>
__device__ __forceinline__ void load_group(u32x4 (&d)[GroupShape<S>::kRows], const char* base, uint32_t lane) {
  const uint32_t v = vec_of_lane<S>(lane);
#pragma unroll
  for (int u = 0; u < GroupShape<S>::kRows; ++u) d[u] = ld_stream(base + 16 * (64 * u + v));
}

template <class S>
__device__ __forceinline__ void store_group(char* base, const u32x4 (&d)[GroupShape<S>::kRows], uint32_t lane) {
  const uint32_t v = vec_of_lane<S>(lane);
#pragma unroll
  for (int u = 0; u < GroupShape<S>::kRows; ++u) st_stream(base + 16 * (64 * u + v), d[u]);
}

// Calls body(vbase, d, lane) for every full row group of the launch, where vbase is the
// group's global vector index and d its data, and stores what the body leaves in d. One
// wave per chunk walks the chunk's groups in address order with the loads of the next AHEAD
// groups in flight while the body works on the current one (each wave streams up to 32 KiB,
// reads and writes interleaved). A wave's chunk indices increase, so its segment cursor
// only moves forward. PACE > 0 (two ahead only): each step of three groups first waits until
// at most PACE memory operations of the wave are outstanding: with 2, only the step's own
// prefetch; with 4, also the previous step's last stores. The lightest sweeps stream HBM
// faster paced (OPT-13B bf16 perturb: 6.40 TB/s with every request the loop allows in
// flight, 6.67 paced at 2, 6.76 at 4; pacing at 6 or 8 measured lower), heavier ones need
// the overlap.
// prologue() runs once per wave, after the loads of the wave's first group are issued (at
// once for a wave without chunks), so that work such as building the update's LDS tables
// overlaps their latency; it may hold a workgroup barrier, which every wave reaches once.
template <class S, int AHEAD, int N, int PACE = 0, class Body, class Prologue>
__device__ __forceinline__ void for_each_group(const Plans<N>& ps, Body body, Prologue prologue) {
  static_assert(PACE == 0 || (AHEAD == 2 && PACE >= 2 && PACE < 16), "pacing applies to the two-ahead loop");
  static_assert(AHEAD == 1 || AHEAD == 2, "one or two groups in flight");
  using G = GroupShape<S>;
  const uint32_t n_waves = gridDim.x * kWavesPerBlock;
  const uint32_t total = ps.chunk_end[ps.count - 1];
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t cg = ps.chunk_groups;
  uint32_t s = 0;
  uint32_t c = blockIdx.x * kWavesPerBlock + wave;
  if (c >= total) prologue();
  for (bool first = true; c < total; c += n_waves, first = false) {
    if (c >= ps.chunk_end[s]) s = segment_of(ps.chunk_end, s + 1, ps.count, c);
    const Plan& pl = ps.p[s];
    // the chunk's groups [g0, g1), relative to the segment's first full group (a select on the
    // chunk index, not a clamped subtraction, which has no scalar form)
    const uint32_t j = c - (s ? ps.chunk_end[s - 1] : 0);
    const uint32_t end = (j + 1) * cg - pl.head;
    const uint32_t g0 = j ? j * cg - pl.head : 0u;
    const uint32_t g1 = end < pl.span ? end : pl.span;
    const uint64_t g_base = pl.g_lo;
    char* base = pl.gbase + static_cast<uint64_t>(g0) * G::kBytes;
    // Rotating register sets: while the body works on one group, the loads of the next AHEAD
    // groups are in flight. No register of an outstanding load is ever copied, and inside the
    // loops the prefetches do not depend on a branch (either would make the compiler wait
    // for every outstanding load before the work).
    u32x4 x[G::kRows], y[G::kRows], z[G::kRows];
    auto work = [&](u32x4 (&cur)[G::kRows], uint32_t g) {
      body((g_base + g) * G::kVecs, cur, lane);
      store_group<S>(base, cur, lane);
      base += G::kBytes;
    };
    auto prefetch = [&](u32x4 (&nxt)[G::kRows], uint32_t ahead) {
      load_group<S>(nxt, base + ahead * G::kBytes, lane);
      __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the work (the scheduler sinks it)
    };
    load_group<S>(x, base, lane);
    if (first) prologue();
    uint32_t g = g0;
    // Each steady-state loop is entered only after one full step of it has run (peeled), so
    // that the loop is entered with the same loads and stores outstanding as its back edge:
    // the compiler then waits for exactly the group a step needs. Entered straight from the
    // first loads, it would merge the two states and wait, in every step, until only the
    // newest loads were outstanding (previous stores and later prefetches included).
    if constexpr (AHEAD == 1) {
      auto step2 = [&]() {
        prefetch(y, 1);
        work(x, g);
        prefetch(x, 1);
        work(y, g + 1);
        g += 2;
      };
      if (g + 2 < g1) {  // at least three groups left: steps of two that both prefetch
        step2();
        while (g + 2 < g1) step2();
      }
      if (g + 1 < g1) {  // two groups left
        prefetch(y, 1);
        work(x, g);
        work(y, g + 1);
      } else {
        work(x, g);
      }
    } else {
      auto step3 = [&]() {
        prefetch(z, 2);
        if constexpr (PACE > 0) __builtin_amdgcn_s_waitcnt(wait_vmcnt(PACE));
        work(x, g);
        prefetch(x, 2);
        work(y, g + 1);
        prefetch(y, 2);
        work(z, g + 2);
        g += 3;
      };
      // 2 to 4 groups left, x and y requested
      auto last = [&]() {
        if (g + 2 < g1) {
          prefetch(z, 2);
          work(x, g);
          if (g + 3 < g1) {
            prefetch(x, 2);
            work(y, g + 1);
            work(z, g + 2);
            work(x, g + 3);
          } else {
            work(y, g + 1);
            work(z, g + 2);
          }
        } else {
          work(x, g);
          work(y, g + 1);
        }
      };
      if (g + 4 < g1) {  // at least five groups left: steps of three that prefetch two ahead
        load_group<S>(y, base + G::kBytes, lane);
        step3();
        while (g + 4 < g1) step3();
        last();
      } else if (g + 1 < g1) {
        load_group<S>(y, base + G::kBytes, lane);
        last();
      } else {
        work(x, g);
      }
    }
  }
}

// Calls body(plan, tile) for every edge tile of the launch, one lane per tile.
template <int N, class Body>
__device__ __forceinline__ void for_each_edge(const Plans<N>& ps, Body body) {
  const uint32_t n_edge = ps.edge_end[ps.count - 1];
  const uint32_t stride = gridDim.x * kBlock;
  for (uint32_t j = blockIdx.x * kBlock + threadIdx.x; j < n_edge; j += stride) {
    const uint32_t s = segment_of(ps.edge_end, 0, ps.count, j);
    const Plan& pl = ps.p[s];
    const uint32_t lj = j - (s ? ps.edge_end[s - 1] : 0);
    body(pl, lj < pl.head_nt ? pl.head_t0 + lj : pl.tail_t0 + (lj - pl.head_nt));
  }
}

// ---------------------------------------------------------------------------------------
// perturb: theta + eps * z_k (bit k mod 8 of each probe byte of group k / 8). TWO: the
// fused transition theta + (eps_a z_a + eps_b z_b), the pair's sum rounded to fp32 first.
struct Probe {
  uint32_t group, bit;
  float eps;
  __device__ __forceinline__ float delta(uint32_t byte) const { return ((byte >> bit) & 1u) ? eps : -eps; }
};

template <class S, bool TWO, int N, int PACE>
__global__ __launch_bounds__(kBlock) void perturb_kernel(Plans<N> ps, Gen gen, Probe a, Probe b) {
  extern __shared__ uint32_t occupancy_pad[];  // dynamic LDS only limits workgroups per CU
  if (ps.count == 0xFFFFFFFFu) occupancy_pad[threadIdx.x] = 0;  // never taken (count <= 64)
  constexpr int R = GroupShape<S>::kRows;
  const bool shared_group = a.group == b.group;
  auto no_prologue = []() {};
  for_each_group<S, 2, N, PACE>(ps, [&](uint64_t vbase, u32x4 (&d)[R], uint32_t lane) {
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
        float dv = a.delta(elem_byte<S>(Wa[u], e));
        if (TWO) dv = dv + b.delta(elem_byte<S>(Wb[u], e));
        v[e] = v[e] + dv;
      }
      d[u] = S::pack(v);
    }
  }, no_prologue);
  for_each_edge(ps, [&](const Plan& pl, uint64_t t) {
    const uint4 ra = gen.block(t, a.group);
    const uint4 rb = TWO ? gen.block(t, b.group) : ra;
    const uint32_t xa[4] = {ra.x, ra.y, ra.z, ra.w}, xb[4] = {rb.x, rb.y, rb.z, rb.w};
    tile_elementwise<S>(reinterpret_cast<typename S::storage*>(pl.base), pl.lo, pl.hi, t, [&](int e, float v) {
      float dv = a.delta(word_byte(xa[e >> 2], e & 3));
      if (TWO) dv = dv + b.delta(word_byte(xb[e >> 2], e & 3));
      return v + dv;
    });
  });
}

// ---------------------------------------------------------------------------------------
// update: theta - lr * sum_k c_k z_k.
struct Coefs {
  float c[ZO_K_MAX];
};

// Spread tables, for streaming launches: C = 32 or 16 copies of each 256-entry table of up to
// 64 / C groups (64 KiB), interleaved so that copy r of entry e of group g is float
// 64 e + C g + r. Lane l reads copy l mod C, which sits in LDS bank (C g + l mod C) mod 32:
// with 32 copies every lane of a half-wave has its own bank, so a 64-lane read of random
// bytes takes 2 LDS cycles instead of about 6.3 when all lanes share one copy; with 16 copies
// two lanes share a bank, about 4 cycles. A lookup's byte address, 256 e + 4 (l mod C) + 4 C g,
// is one byte permute of the generator word and the lane's copy offset (as many instructions
// as a lookup into a shared table).
constexpr uint32_t kSpreadFloats = 256 * 64;
// floats of the tables of NG groups: C interleaved copies, or one shared copy (C = 0)
template <int NG, int C>
constexpr uint32_t table_floats() {
  static_assert(C == 0 || (C == 16 || C == 32) && NG * C <= 64, "spread tables fill at most 64 KiB");
  return C == 0 ? NG * 256 : kSpreadFloats;
}

// Build the n_groups x 256 table in LDS (C > 0: the interleaved copies). Entry (g, b):
// fl(lr * t), t the sum over the group's 8 probe slots of +-c (bit set: +c), pairwise; slots
// outside [k_base, k_base + K) contribute 0. Scaling each entry once here saves the sweep a
// multiply per element; with one probe the entry is +-fl(lr * c), the step a perturb by
// -fl(lr * c) would apply. Thread b writes entry b of every group: the group loop and the
// coefficient reads are uniform (scalar loads), and the sign of slot s is an XOR of the
// coefficient's sign bit with bit s of ~b.
static_assert(kBlock == 256, "one table entry per thread");
template <int C>
__device__ __forceinline__ void build_tables(float* tab, const Coefs& cf, uint32_t k_base, uint32_t K,
                                             uint32_t n_groups, float lr) {
  const uint32_t b = threadIdx.x;
  uint32_t flip[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) flip[s] = ((~b) << (31 - s)) & 0x80000000u;
  const uint32_t g_first = k_base / 8;
  for (uint32_t g = 0; g < n_groups; ++g) {
    float v[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint32_t k = 8u * (g_first + g) + s;
      const float cv = (k >= k_base && k - k_base < K) ? cf.c[k - k_base] : 0.0f;
      v[s] = __uint_as_float(__float_as_uint(cv) ^ flip[s]);
    }
    const float t = (((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]))) * lr;
    if constexpr (C > 0) {
      // entry b's C / 4 float4 of copies, 256 bytes after entry b - 1's: thread b writes them
      // starting at float4 b mod (C / 4), so that the lanes of each write spread over the banks
      // the group's copies occupy (in a fixed order all 64 would land on the same 4 banks)
      constexpr uint32_t Q = C / 4;
      float* e = tab + 64u * b + C * g;
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
// lane's copy offset `lane_off` = 4 (l mod C), byte 1: byte e of w, upper bytes 0), then the
// float there plus the group's offset 4 C g.
template <int C>
__device__ __forceinline__ float spread_at(const float* tab, uint32_t lane_off, uint32_t w, int e, uint32_t g) {
  const uint32_t addr = __builtin_amdgcn_perm(w, lane_off, 0x0C0C0000u | ((4u + static_cast<uint32_t>(e)) << 8));
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(tab) + addr + 4u * C * g);
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
// at compile time (one run) and leaves the last group's generator words in Wlast; NG == 0:
// runs of 8 groups, Neumaier-compensated across runs (Wlast is not written).
template <class S, int NG, int C>
__device__ __forceinline__ void group_sums(float (&acc)[GroupShape<S>::kRows][S::kVecElems], const float* tab,
                                           const Gen& gen, uint64_t vbase, uint32_t lane, uint32_t n_groups,
                                           uint32_t g_first, uint32_t lane_off,
                                           uint32_t (&Wlast)[GroupShape<S>::kRows][S::kWords]) {
  constexpr int R = GroupShape<S>::kRows;
  static_assert(C == 0 || NG > 0, "spread tables need a fixed group count");
  if constexpr (NG > 0) {
    add_group<S, true, C>(acc, tab, gen, vbase, lane, 0, g_first, lane_off, Wlast);
#pragma unroll
    for (int g = 1; g < NG; ++g)
      add_group<S, false, C>(acc, tab, gen, vbase, lane, g, g_first, lane_off, Wlast);
  } else {
    float comp[R][S::kVecElems];
    uint32_t W[R][S::kWords];
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
      const uint4 r = gen.block(t, g_first + g);
      const uint32_t x[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int j = 0; j < (int)kTile; ++j) {
        const uint32_t byte = word_byte(x[j >> 2], j & 3);
        float v;
        if constexpr (C > 0) {
          v = tab[64u * byte + C * g + (threadIdx.x % C)];
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

// RESTORE: theta + eps_r z_r - lr * sum (the last probe's restore merged with the update):
// t = fl(theta + delta_r), then t minus the sum of the lr-scaled table values. When the count of
// groups is fixed and the restore probe lies in the last of them (Algorithm 1 restores the
// step's last probe), its generator words are those the group sum has just produced; otherwise
// they are generated after the group loop (keeping a middle group's words would hold them live
// across the rest of it).
template <class S, int NG, bool RESTORE, int N, int C>
__global__ __launch_bounds__(kBlock) void update_kernel(Plans<N> ps, Gen gen, uint32_t k_base, uint32_t K,
                                                       uint32_t n_groups, Coefs cf, float lr, Probe r) {
  // n_groups x 256 floats (C > 0: the interleaved copies): static for a fixed group count
  // (constant LDS offsets), else dynamic.
  extern __shared__ float tab_dyn[];
  __shared__ float tab_fix[NG > 0 ? table_floats<NG, C>() : 1];
  float* tab = NG > 0 ? tab_fix : tab_dyn;
  // the tables are built while each wave's first loads are in flight (for_each_group's prologue)
  auto build = [&]() { build_tables<C>(tab, cf, k_base, K, n_groups, lr); };
  const uint32_t lane_off = 4u * (threadIdx.x % (C > 0 ? C : 32));  // the lane's copy of a spread table
  const uint32_t g_first = k_base / 8;
  constexpr int R = GroupShape<S>::kRows;
  // two groups in flight for the table counts that stream at one or two workgroups per CU;
  // one for the heavier updates, which run more waves per CU
  constexpr int kAhead = C > 0 || NG == 1 || NG == 2 || NG == 4 ? 2 : 1;
  const bool restore_in_last = NG > 0 && r.group == g_first + static_cast<uint32_t>(NG) - 1;  // uniform
  for_each_group<S, kAhead, N>(ps, [&](uint64_t vbase, u32x4 (&d)[R], uint32_t lane) {
    float acc[R][S::kVecElems];
    uint32_t Wr[R][S::kWords];  // the last group's words, then the restore probe's
    group_sums<S, NG, C>(acc, tab, gen, vbase, lane, n_groups, g_first, lane_off, Wr);
    if (RESTORE && !restore_in_last) group_words(gen, vbase, lane, r.group, Wr, S());
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float v[S::kVecElems];
      S::unpack(d[u], v);
#pragma unroll
      for (int e = 0; e < S::kVecElems; ++e) {
        if (RESTORE) v[e] = v[e] + r.delta(elem_byte<S>(Wr[u], e));
        v[e] = v[e] - acc[u][e];
      }
      d[u] = S::pack(v);
    }
  }, build);
  for_each_edge(ps, [&](const Plan& pl, uint64_t t) {
    float acc[kTile];
    tile_sums<C>(acc, tab, gen, t, n_groups, g_first);
    const uint4 rr = RESTORE ? gen.block(t, r.group) : make_uint4(0, 0, 0, 0);
    const uint32_t xr[4] = {rr.x, rr.y, rr.z, rr.w};
    tile_elementwise<S>(reinterpret_cast<typename S::storage*>(pl.base), pl.lo, pl.hi, t, [&](int e, float v) {
      if (RESTORE) v = v + r.delta(word_byte(xr[e >> 2], e & 3));
      return v - acc[e];
    });
  });
}

// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void gen_bits_kernel(uint8_t* out, uint64_t tile_begin, uint64_t n_tiles,
                                                         uint32_t group, Gen gen) {
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n_tiles; i += stride) {
    const uint4 r = gen.block(tile_begin + i, group);
    *reinterpret_cast<u32x4*>(out + 16 * i) = u32x4{r.x, r.y, r.z, r.w};
  }
}

// ---------------------------------------------------------------------------------------
// Host side.
constexpr int kSegsPerLaunch = 64;                 // segments per batched launch (kernel arguments, ~5 KiB)
constexpr uint64_t kMaxLaunchChunks = 1ull << 31;  // chunks per launch: 32-bit indices with room for the stride

// The grid's cap: zo_set_max_blocks if set, else kDefaultMaxBlocks, or (sized) none: the
// caller then sized work_items per workgroup itself.
uint32_t cap_blocks(bool sized = false) { return g_max_blocks ? g_max_blocks : sized ? (1u << 30) : kDefaultMaxBlocks; }

uint32_t grid_for(uint64_t work_items, uint64_t per_block, bool sized = false) {
  const uint64_t need = (work_items + per_block - 1) / per_block;
  const uint64_t cap = cap_blocks(sized);
  const uint64_t g = need < cap ? need : cap;
  return static_cast<uint32_t>(g ? g : 1);
}

int check_params(const void* params, zo_dtype dt, uint64_t offset, uint64_t n) {
  if (dt != ZO_F32 && dt != ZO_BF16) return ZO_ERR_ARG;
  if (n == 0) return ZO_OK;
  if (params == nullptr) return ZO_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(params) % (dt == ZO_F32 ? 4 : 2) != 0) return ZO_ERR_ARG;
  if (offset + n < offset || offset + n == 0) return ZO_ERR_ARG;  // reaches 2^64
  if (n >= ZO_N_MAX) return ZO_ERR_ARG;  // more weights than a device holds
  return ZO_OK;
}

uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

// Full row groups need the address of global element 0 (params shifted back by offset
// elements) to be 16-byte aligned, so that every group vector is an aligned 16 bytes.
Plan make_plan(void* params, uint64_t offset, uint64_t n, size_t elem, uint32_t chunk_groups) {
  Plan pl{};
  pl.base = static_cast<char*>(params);
  pl.lo = offset;
  pl.hi = offset + n;
  if (n == 0) return pl;
  const uintptr_t base = reinterpret_cast<uintptr_t>(params) - static_cast<uintptr_t>(offset * elem);
  uint64_t head_end = pl.hi, tail_begin = pl.hi;
  if ((base & 15u) == 0) {
    const uint64_t g_lo = ceil_div(pl.lo, kGroupElems), g_hi = pl.hi / kGroupElems;
    if (g_lo < g_hi) {  // g_hi - g_lo < 2^30: n < ZO_N_MAX is checked first
      pl.g_lo = g_lo;
      pl.span = static_cast<uint32_t>(g_hi - g_lo);
      pl.head = static_cast<uint32_t>(g_lo % chunk_groups);
      pl.gbase = pl.base + (g_lo * kGroupElems - pl.lo) * elem;
      head_end = g_lo * kGroupElems;
      tail_begin = g_hi * kGroupElems;
    }
  }
  if (head_end > pl.lo) {
    pl.head_t0 = pl.lo / kTile;
    pl.head_nt = static_cast<uint32_t>(ceil_div(head_end, kTile) - pl.head_t0);
  }
  if (pl.hi > tail_begin) {
    pl.tail_t0 = tail_begin / kTile;
    pl.tail_nt = static_cast<uint32_t>(ceil_div(pl.hi, kTile) - pl.tail_t0);
  }
  return pl;
}

// Chunks that meet a plan's full row groups (fewer than 2^30 + 2).
uint32_t plan_chunks(const Plan& pl, uint32_t chunk_groups) {
  return pl.span ? static_cast<uint32_t>(ceil_div(static_cast<uint64_t>(pl.head) + pl.span, chunk_groups)) : 0u;
}

template <int N>
void add_plan(Plans<N>& ps, const Plan& pl) {
  const uint32_t s = ps.count++;
  ps.p[s] = pl;
  ps.chunk_end[s] = (s ? ps.chunk_end[s - 1] : 0) + plan_chunks(pl, ps.chunk_groups);
  ps.edge_end[s] = (s ? ps.edge_end[s - 1] : 0) + pl.head_nt + pl.tail_nt;
}

// chunks_per_wave > 0: one workgroup per kWavesPerBlock * chunks_per_wave chunks; 0: up to
// kDefaultMaxBlocks workgroups, grid-stride beyond.
template <int N>
uint32_t plans_grid(const Plans<N>& ps, uint32_t chunks_per_wave) {
  const uint32_t chunks = ps.chunk_end[ps.count - 1], edges = ps.edge_end[ps.count - 1];
  const uint32_t a =
      chunks ? grid_for(chunks, uint64_t{kWavesPerBlock} * (chunks_per_wave ? chunks_per_wave : 1), chunks_per_wave > 0) : 1;
  const uint32_t b = grid_for(edges, kBlock);
  return a > b ? a : b;
}

int launch_status() { return hipGetLastError() == hipSuccess ? ZO_OK : ZO_ERR_HIP; }

Probe make_probe(uint32_t k, float eps) { return Probe{k / 8, k % 8, eps}; }

Gen make_gen(uint64_t seed, uint32_t step) {
  return Gen{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), step};
}

// What one sweep applies: one or two probes, or the update (with an optional restore probe).
struct Sweep {
  bool update;
  Probe a, b;
  bool two;
  uint32_t k_base, K, n_groups;
  Coefs cf;
  float lr;
  Probe r;
  bool restore;
};

// Streaming shape of a launch over `elements` weights of `elem` bytes. HBM sustains these
// in-place sweeps best as few long sequential read-write streams: each wave walks up to
// kMaxChunkBytes of consecutive row groups with the next one or two groups in flight, and
// occupancy is capped with dynamic LDS so that few waves stream at once (the bf16 perturb on
// an OPT-13B shaped buffer: 6.5 TB/s at one workgroup per CU, 5.6 at full occupancy). An
// update needs more waves where its generator and table work per byte outgrows what one wave
// overlaps with its own loads; the caps below are the fastest of 1-4 workgroups per CU and
// full occupancy, 16 to 64 KiB chunks and one or two groups in flight, measured for every
// kernel on OPT-13B shaped bf16 and 3 G-element fp32 buffers (four bf16 probe groups with
// their 16-copy tables: on an OPT-30B shaped buffer). Updates with more probe groups
// (K >= 40 in bf16, K >= 56 in fp32) are bound by the generator or the LDS table lookups
// and keep 4 KiB chunks at full occupancy, as do sweeps smaller than the 256 MiB Infinity
// Cache. Grids: up to kDefaultMaxBlocks workgroups, grid-stride beyond (in-order dispatch of
// many short-lived workgroups keeps the streams compact; a persistent grid of one workgroup
// per CU measured 5.6 TB/s), except that the one-probe bf16 perturb, the two-probe fp32
// perturb, the one-group bf16 update and the two-group bf16 update with restore run one chunk
// per wave (OPT-13B: the perturb 6.48 -> 6.67 TB/s, OPT-30B 6.20 -> 6.60; 3 G fp32 weights:
// the two-probe perturb 6.14 -> 6.22 in one probe group, 6.30 -> 6.48 across two; OPT-30B
// K = 8: the update 6.19 -> 6.53, with restore 6.41 -> 6.70; OPT-13B K = 16, the update with
// restore 5.94 -> 6.13; the other kernels measured equal or slower so, the K = 16 update 6.41
// against 6.54 TB/s).
struct Shape {
  uint32_t chunk_groups;
  uint32_t blocks_per_cu;    // 0: no cap
  uint32_t chunks_per_wave;  // 0: up to kDefaultMaxBlocks workgroups, grid-stride beyond
};

constexpr uint64_t kStreamBytes = 256ull << 20;

Shape shape_for(uint64_t elements, size_t elem, const Sweep& w) {
  const uint64_t group_bytes = kGroupElems * elem;
  const Shape short_chunks{static_cast<uint32_t>(4096 / group_bytes ? 4096 / group_bytes : 1), 0, 0};
  if (elements * elem < kStreamBytes) return short_chunks;
  uint32_t cap = 1;  // the perturb kernels, one or two probes
  if (w.update) {
    const uint32_t g = w.n_groups;
    if (elem == 2)
      cap = g == 1 ? 1 : g == 2 ? (w.restore ? 2 : 1) : g == 3 ? 3 : g == 4 ? 2 : 0;
    else
      cap = g <= 3 ? 1 : g == 4 ? 2 : g <= 6 ? 3 : 0;
  }
  if (cap == 0) return short_chunks;
  const bool one_probe_bf16 = !w.update && !w.two && elem == 2;
  const bool two_probes_fp32 = !w.update && w.two && elem == 4;
  const bool one_group_update_bf16 = w.update && w.n_groups == 1 && elem == 2;
  const bool restore_two_groups_bf16 = w.update && w.restore && w.n_groups == 2 && elem == 2;
  return Shape{static_cast<uint32_t>(kMaxChunkBytes / group_bytes), cap,
               one_probe_bf16 || two_probes_fp32 || one_group_update_bf16 || restore_two_groups_bf16 ? 1u : 0u};
}

// Dynamic LDS that, with `static_lds` bytes of the kernel's own, admits exactly `cap`
// workgroups on a CU's 160 KiB (0: no cap).
size_t occupancy_lds(uint32_t cap, size_t static_lds) {
  if (cap == 0) return 0;
  const size_t per_block = cap == 1 ? 96 * 1024 : cap == 2 ? 72 * 1024 : cap == 3 ? 48 * 1024 : 36 * 1024;
  return per_block > static_lds ? per_block - static_lds : 0;
}

// A workgroup's LDS above 64 KiB (static plus dynamic) must be allowed per kernel before the
// launch.
template <class K>
void allow_lds(K kernel, size_t dynamic_bytes, size_t static_bytes = 0) {
  if (dynamic_bytes + static_bytes > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(dynamic_bytes));
}

template <class S, int N>
void launch_sweep(const Plans<N>& ps, const Gen& gen, const Sweep& w, const Shape& sh, hipStream_t st) {
  const uint32_t cap = sh.blocks_per_cu;
  const dim3 grid(plans_grid(ps, sh.chunks_per_wave)), block(kBlock);
  if (!w.update) {
    const size_t pad = occupancy_lds(cap, 0);
    auto go = [&](auto kernel, Probe b) {
      allow_lds(kernel, pad);
      kernel<<<grid, block, pad, st>>>(ps, gen, w.a, b);
    };
    // paced when the generator work per byte is lightest: one probe group, or fp32 with two;
    // bf16 at 4 outstanding operations (one probe +1.3%, two in one group +3.4% over 2), fp32
    // at 2 (4 measured equal or lower)
    constexpr int kPace = sizeof(typename S::storage) == 2 ? 4 : 2;
    const bool two_groups = w.two && w.a.group != w.b.group;
    const bool paced = (two_groups ? 2u : 1u) * (sizeof(typename S::storage) == 2 ? 2u : 1u) <= 2u;
    if (w.two)
      paced ? go(perturb_kernel<S, true, N, kPace>, w.b) : go(perturb_kernel<S, true, N, 0>, w.b);
    else
      paced ? go(perturb_kernel<S, false, N, kPace>, w.a) : go(perturb_kernel<S, false, N, 0>, w.a);
    return;
  }
  const bool fixed = w.n_groups == 1 || w.n_groups == 2 || w.n_groups == 4 || w.n_groups == 8;
  // Copies of each table (64 KiB in all), where they measured faster: 32 for two groups (one in
  // fp32) streaming at a capped occupancy (64 KiB per workgroup would limit an uncapped launch
  // to two workgroups per CU; a single bf16 group leaves the shared table's LDS half idle and
  // gains nothing); 16 for four bf16 groups at two workgroups per CU (OPT-30B K = 32: 23.6 ->
  // 22.0 ms against shared tables at full occupancy; 32 copies, 128 KiB at one workgroup per
  // CU, 26.1 ms, and 16 copies of eight groups at one per CU lost a third: four waves per CU
  // cannot hide the generator and table latencies).
  const bool bf16 = sizeof(typename S::storage) == 2;
  uint32_t copies = 0;
  if (cap > 0) {
    if (w.n_groups == 2 || (w.n_groups == 1 && !bf16))
      copies = 32;
    else if (w.n_groups == 4 && bf16)
      copies = 16;
  }
  const size_t table_bytes =
      copies ? size_t{kSpreadFloats} * sizeof(float) : static_cast<size_t>(w.n_groups) * 256 * sizeof(float);
  const size_t static_lds = fixed ? table_bytes : 0;
  const size_t pad = occupancy_lds(cap, static_lds);
  const size_t tables = fixed ? 0 : table_bytes;
  const size_t lds = tables > pad ? tables : pad;  // dynamic tables (up to 128 KiB) or the pad
  auto go = [&](auto kernel) {
    allow_lds(kernel, lds, static_lds);
    kernel<<<grid, block, lds, st>>>(ps, gen, w.k_base, w.K, w.n_groups, w.cf, w.lr, w.r);
  };
  auto dispatch = [&](auto restore) {
    constexpr bool R = decltype(restore)::value;
    switch (w.n_groups) {
      case 1: copies ? go(update_kernel<S, 1, R, N, 32>) : go(update_kernel<S, 1, R, N, 0>); break;
      case 2: copies ? go(update_kernel<S, 2, R, N, 32>) : go(update_kernel<S, 2, R, N, 0>); break;
      case 4: copies ? go(update_kernel<S, 4, R, N, 16>) : go(update_kernel<S, 4, R, N, 0>); break;
      case 8: go(update_kernel<S, 8, R, N, 0>); break;
      default: go(update_kernel<S, 0, R, N, 0>); break;
    }
  };
  if (w.restore)
    dispatch(std::true_type{});
  else
    dispatch(std::false_type{});
}

int check_sweep(const Sweep& w) {
  if (!std::isfinite(w.a.eps) || (w.two && !std::isfinite(w.b.eps))) return ZO_ERR_NONFINITE;
  if (w.update && (!std::isfinite(w.lr) || (w.restore && !std::isfinite(w.r.eps)))) return ZO_ERR_NONFINITE;
  return ZO_OK;
}

int make_update_sweep(Sweep& w, uint32_t k_base, uint32_t K, const float* c, float lr, const Probe* r) {
  if (K > ZO_K_MAX) return ZO_ERR_ARG;
  if (static_cast<uint64_t>(k_base) + K > (1ull << 32)) return ZO_ERR_ARG;
  if (K > 0 && c == nullptr) return ZO_ERR_NULL;
  if (!std::isfinite(lr) || (r && !std::isfinite(r->eps))) return ZO_ERR_NONFINITE;
  for (uint32_t j = 0; j < K; ++j)
    if (!std::isfinite(c[j])) return ZO_ERR_NONFINITE;
  w = Sweep{};
  if (K == 0) {  // nothing to sum: the restore alone, or nothing
    w.update = false;
    w.a = r ? *r : Probe{0, 0, 0.0f};
    return ZO_OK;
  }
  w.update = true;
  for (uint32_t j = 0; j < ZO_K_MAX; ++j) w.cf.c[j] = j < K ? c[j] : 0.0f;
  w.k_base = k_base;
  w.K = K;
  const uint32_t g_first = k_base / 8;
  const uint32_t g_last = static_cast<uint32_t>((static_cast<uint64_t>(k_base) + K - 1) / 8);
  w.n_groups = g_last - g_first + 1;
  w.lr = lr;
  w.restore = r != nullptr && r->eps != 0.0f;  // a zero restore changes nothing (theta + 0 = theta)
  w.r = r ? *r : Probe{0, 0, 0.0f};
  return ZO_OK;
}

// One contiguous tensor.
template <class S>
int run_one(void* params, uint64_t offset, uint64_t n, uint64_t seed, uint32_t step, const Sweep& w, void* stream) {
  const Shape sh = shape_for(n, sizeof(typename S::storage), w);
  Plans<1> ps{};
  ps.chunk_groups = sh.chunk_groups;
  add_plan(ps, make_plan(params, offset, n, sizeof(typename S::storage), sh.chunk_groups));
  (void)hipGetLastError();
  launch_sweep<S>(ps, make_gen(seed, step), w, sh, static_cast<hipStream_t>(stream));
  return launch_status();
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

// A list of tensors: validated as a whole (alignment, index ranges, no two segments sharing
// memory), then swept in launches of up to kSegsPerLaunch segments.
int check_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype) {
  if (dtype != ZO_F32 && dtype != ZO_BF16) return ZO_ERR_ARG;
  if (n_segs == 0) return ZO_OK;
  if (segs == nullptr) return ZO_ERR_NULL;
  const size_t elem = dtype == ZO_F32 ? 4 : 2;
  std::vector<std::pair<uintptr_t, uintptr_t>> spans;
  spans.reserve(n_segs);
  for (uint32_t i = 0; i < n_segs; ++i) {
    const int rc = check_params(segs[i].params, dtype, segs[i].offset, segs[i].n);
    if (rc != ZO_OK) return rc;
    if (segs[i].n == 0) continue;
    const uintptr_t a = reinterpret_cast<uintptr_t>(segs[i].params);
    if (segs[i].n > (UINTPTR_MAX - a) / elem) return ZO_ERR_ARG;
    spans.emplace_back(a, a + segs[i].n * elem);
  }
  std::sort(spans.begin(), spans.end());
  for (size_t i = 1; i < spans.size(); ++i)
    if (spans[i].first < spans[i - 1].second) return ZO_ERR_ARG;  // overlapping memory
  return ZO_OK;
}

template <class S>
int run_segments(const zo_segment* segs, uint32_t n_segs, uint64_t seed, uint32_t step, const Sweep& w,
                 void* stream) {
  const Gen gen = make_gen(seed, step);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t total = 0;  // the call's weights decide the streaming shape of all its launches
  for (uint32_t i = 0; i < n_segs; ++i) total += segs[i].n;
  const Shape sh = shape_for(total, sizeof(typename S::storage), w);
  (void)hipGetLastError();
  Plans<kSegsPerLaunch> ps{};
  ps.chunk_groups = sh.chunk_groups;
  for (uint32_t i = 0; i < n_segs; ++i) {
    if (segs[i].n == 0) continue;
    const Plan pl = make_plan(segs[i].params, segs[i].offset, segs[i].n, sizeof(typename S::storage), sh.chunk_groups);
    if (ps.count && ps.chunk_end[ps.count - 1] + static_cast<uint64_t>(plan_chunks(pl, sh.chunk_groups)) >= kMaxLaunchChunks) {
      launch_sweep<S>(ps, gen, w, sh, st);  // keep a launch's chunk count 32-bit
      if (launch_status() != ZO_OK) return ZO_ERR_HIP;
      ps.count = 0;
    }
    add_plan(ps, pl);
    if (ps.count == kSegsPerLaunch) {
      launch_sweep<S>(ps, gen, w, sh, st);
      if (launch_status() != ZO_OK) return ZO_ERR_HIP;
      ps.count = 0;
    }
  }
  if (ps.count) {
    launch_sweep<S>(ps, gen, w, sh, st);
    return launch_status();
  }
  return ZO_OK;
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

Sweep perturb_sweep(uint32_t k_a, float eps_a, const uint32_t* k_b, float eps_b) {
  Sweep w{};
  w.a = make_probe(k_a, eps_a);
  w.two = k_b != nullptr;
  w.b = k_b ? make_probe(*k_b, eps_b) : w.a;
  return w;
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
  gen_bits_kernel<<<dim3(grid_for(n_tiles, kBlock)), dim3(kBlock), 0, static_cast<hipStream_t>(stream)>>>(
      out_dev, tile_begin, n_tiles, group, make_gen(seed, step));
  return launch_status();
}

void zo_set_max_blocks(uint32_t max_blocks) { g_max_blocks = max_blocks; }

}  // extern "C"
