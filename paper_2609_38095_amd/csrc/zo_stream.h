// Streaming loops of libzo's sweeps for gfx950 (CDNA4), shared by the probe sweeps
// (zo_sweep.hip) and the plain read-modify-write ceiling (calib/rmw_ceiling.hip), so that the
// ceiling walks memory exactly as the sweeps do.
//
// Memory layout of a sweep. theta is walked in row groups of 1024 elements: 2 (bf16) or 4
// (fp32) rows of 64 contiguous 16-byte vectors, one vector per lane and row, so each load and
// store instruction of a wave covers 1 KiB of contiguous memory (non-temporal: nothing is
// reused). A tile of 16 elements spans 2 vectors (bf16) or 4 (fp32); the lanes holding one
// tile are m and m + 32 (bf16) or m, m + 16, m + 32, m + 48 (fp32), which lets the probe
// sweeps hand generator words between them with the gfx950 half-wave swaps. A wave streams a
// chunk of consecutive row groups (up to 32 KiB) with the loads of the next one, two or three
// groups in flight while it works on the current one. The loops are written so that the
// compiler's memory waits are exact, and can be paced explicitly. Head and tail elements that
// do not fill a row group (and everything, when the storage is not 16-byte aligned relative to
// the global index) take an element-wise path, one tile per lane.
#ifndef ZO_STREAM_H_
#define ZO_STREAM_H_

#include <hip/hip_runtime.h>

#include <cstdint>

#include "zo_plan.h"

namespace zo {

// s_waitcnt immediate for vmcnt(n), n < 16, that leaves expcnt and lgkmcnt unconstrained
// (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int wait_vmcnt(int n) { return 0x0F70 | n; }

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
// group's global vector index and d its data, and stores what the body leaves in d. Each
// chunk is one stream walked in address order by WPS waves of a workgroup of BLOCK threads:
// wave w of the stream takes the chunk's groups w, w + WPS, w + 2 WPS, ..., with the loads of
// its next AHEAD groups in flight while the body works on the current one (a stream of up to
// 32 KiB, reads and writes interleaved). More waves per stream give the generator and table
// work more waves to hide behind without adding streams. A wave's chunk indices increase,
// so its segment cursor only moves forward. PACE > 0 (two or three ahead): each step of
// the loop first waits until at most PACE memory operations of the wave are outstanding:
// two ahead, with 2 only the step's own prefetch, with 4 also the previous step's last
// stores. The lighter sweeps stream HBM faster paced (OPT-13B bf16 perturb: 6.40 TB/s with
// every request the loop allows in flight, 6.67 paced at 2, 6.76 at 4; pacing at 6 or 8
// measured lower; the one- and two-group bf16 updates +0.3-0.5% at 4), heavier ones need the
// overlap.
// prologue() runs once per wave, after the loads of the wave's first group are issued (at
// once for a wave without groups), so that work such as building the update's LDS tables
// overlaps their latency; it may hold a workgroup barrier, which every wave reaches once.
template <class S, int AHEAD, int N, int PACE = 0, int BLOCK = 256, int WPS = 1, class Body, class Prologue>
__device__ __forceinline__ void for_each_group(const Plans<N>& ps, Body body, Prologue prologue) {
  static_assert(PACE == 0 || (AHEAD >= 2 && PACE >= 2 && PACE < 16), "pacing applies to the two- and three-ahead loops");
  static_assert(AHEAD >= 1 && AHEAD <= 3, "one to three groups in flight");
  static_assert(BLOCK % 64 == 0 && (WPS == 1 || WPS == 2 || WPS == 4) && (BLOCK / 64) % WPS == 0,
                "whole streams per workgroup");
  using G = GroupShape<S>;
  constexpr uint32_t kStreams = BLOCK / 64 / WPS;  // streams per workgroup
  constexpr uint64_t kStride = WPS * G::kBytes;    // bytes between one wave's groups
  const uint32_t n_streams = gridDim.x * kStreams;
  const uint32_t total = ps.chunk_end[ps.count - 1];
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t sub = wave % WPS;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t cg = ps.chunk_groups;
  uint32_t s = 0;
  uint32_t c = blockIdx.x * kStreams + wave / WPS;
  if (c >= total) prologue();
  for (bool first = true; c < total; c += n_streams, first = false) {
    if (c >= ps.chunk_end[s]) s = segment_of(ps.chunk_end, s + 1, ps.count, c);
    const Plan& pl = ps.p[s];
    // slot j of the segment holds groups [j cg - head, (j + 1) cg - head) clipped to [0, span)
    // (relative to the segment's first full group); leading alignment slots hold none
    const uint32_t j = c - (s ? ps.chunk_end[s - 1] : 0);
    const uint32_t a = j * cg, b = (j + 1) * cg, top = pl.head + pl.span;
    const uint32_t lo = a > pl.head ? a : pl.head, hi = b < top ? b : top;
    if (lo + sub >= hi) {  // an alignment slot, or a short chunk without a group for this wave
      if (first) prologue();
      continue;
    }
    const uint32_t g0 = lo - pl.head + sub;  // this wave's first group
    const uint32_t g1 = hi - pl.head;
    const uint32_t cnt = (g1 - g0 + (WPS - 1)) / WPS;  // this wave's groups in the chunk
    const uint64_t g_base = pl.g_lo;
    char* base = pl.gbase + static_cast<uint64_t>(g0) * G::kBytes;
    // Rotating register sets: while the body works on one group, the loads of the next AHEAD
    // groups are in flight. No register of an outstanding load is ever copied, and inside the
    // loops the prefetches do not depend on a branch (either would make the compiler wait
    // for every outstanding load before the work).
    u32x4 x[G::kRows], y[G::kRows], z[G::kRows], v[G::kRows];
    uint32_t g = g0, i = 0;  // the current group and its index among the wave's groups
    auto work = [&](u32x4 (&cur)[G::kRows]) {
      body((g_base + g) * G::kVecs, cur, lane);
      store_group<S>(base, cur, lane);
      base += kStride;
      g += WPS;
      ++i;
    };
    auto prefetch = [&](u32x4 (&nxt)[G::kRows], uint32_t ahead) {
      load_group<S>(nxt, base + ahead * kStride, lane);
      __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the work (the scheduler sinks it)
    };
    load_group<S>(x, base, lane);
    if (first) prologue();
    // Each steady-state loop is entered only after one full step of it has run (peeled), so
    // that the loop is entered with the same loads and stores outstanding as its back edge:
    // the compiler then waits for exactly the group a step needs. Entered straight from the
    // first loads, it would merge the two states and wait, in every step, until only the
    // newest loads were outstanding (previous stores and later prefetches included).
    if constexpr (AHEAD == 1) {
      auto step2 = [&]() {
        prefetch(y, 1);
        work(x);
        prefetch(x, 1);
        work(y);
      };
      if (i + 2 < cnt) {  // at least three groups left: steps of two that both prefetch
        step2();
        while (i + 2 < cnt) step2();
      }
      if (i + 1 < cnt) {  // two groups left
        prefetch(y, 1);
        work(x);
        work(y);
      } else {
        work(x);
      }
    } else if constexpr (AHEAD == 2) {
      auto step3 = [&]() {
        prefetch(z, 2);
        if constexpr (PACE > 0) __builtin_amdgcn_s_waitcnt(wait_vmcnt(PACE));
        work(x);
        prefetch(x, 2);
        work(y);
        prefetch(y, 2);
        work(z);
      };
      // 2 to 4 groups left, x and y requested
      auto last = [&]() {
        if (i + 2 < cnt) {
          prefetch(z, 2);
          work(x);
          if (i + 2 < cnt) {
            prefetch(x, 2);
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
      if (i + 4 < cnt) {  // at least five groups left: steps of three that prefetch two ahead
        load_group<S>(y, base + kStride, lane);
        step3();
        while (i + 4 < cnt) step3();
        last();
      } else if (i + 1 < cnt) {
        load_group<S>(y, base + kStride, lane);
        last();
      } else {
        work(x);
      }
    } else {
      auto step4 = [&]() {
        prefetch(v, 3);
        if constexpr (PACE > 0) __builtin_amdgcn_s_waitcnt(wait_vmcnt(PACE));
        work(x);
        prefetch(x, 3);
        work(y);
        prefetch(y, 3);
        work(z);
        prefetch(z, 3);
        work(v);
      };
      // 3 to 6 groups left, x, y and z requested
      auto last = [&]() {
        if (i + 3 < cnt) {
          prefetch(v, 3);
          work(x);
          if (i + 3 < cnt) {
            prefetch(x, 3);
            work(y);
            if (i + 3 < cnt) {
              prefetch(y, 3);
              work(z);
              work(v);
              work(x);
              work(y);
            } else {
              work(z);
              work(v);
              work(x);
            }
          } else {
            work(y);
            work(z);
            work(v);
          }
        } else {
          work(x);
          work(y);
          work(z);
        }
      };
      if (i + 6 < cnt) {  // at least seven groups left: steps of four that prefetch three ahead
        load_group<S>(y, base + kStride, lane);
        load_group<S>(z, base + 2 * kStride, lane);
        step4();
        while (i + 6 < cnt) step4();
        last();
      } else if (i + 2 < cnt) {
        load_group<S>(y, base + kStride, lane);
        load_group<S>(z, base + 2 * kStride, lane);
        last();
      } else if (i + 1 < cnt) {
        load_group<S>(y, base + kStride, lane);
        work(x);
        work(y);
      } else {
        work(x);
      }
    }
  }
}

// Calls body(plan, tile) for every edge tile of the launch, one lane per tile.
template <int N, int BLOCK, class Body>
__device__ __forceinline__ void for_each_edge(const Plans<N>& ps, Body body) {
  const uint32_t n_edge = ps.edge_end[ps.count - 1];
  const uint32_t stride = gridDim.x * BLOCK;
  for (uint32_t j = blockIdx.x * BLOCK + threadIdx.x; j < n_edge; j += stride) {
    const uint32_t s = segment_of(ps.edge_end, 0, ps.count, j);
    const Plan& pl = ps.p[s];
    const uint32_t lj = j - (s ? ps.edge_end[s - 1] : 0);
    body(pl, lj < pl.head_nt ? pl.head_t0 + lj : pl.tail_t0 + (lj - pl.head_nt));
  }
}

}  // namespace zo

#endif  // ZO_STREAM_H_
