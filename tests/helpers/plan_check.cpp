// Host checker of libzo's launch planning, validation and coefficient code, built with
// AddressSanitizer and UBSan by tests/test_host_sanitized.py (g++, no GPU). It replays on the
// CPU the index arithmetic the sweep kernels do with what the planner hands them, and checks
// that every element of every tensor is covered exactly once:
//   - make_plan: head tiles, full row groups and tail tiles partition [offset, offset + n),
//     for element sizes 2 and 4, aligned and unaligned bases, offsets up to the top of the
//     64-bit index range and n up to ZO_N_MAX - 1;
//   - the chunk walk of the kernels (32-bit chunk and group indices relative to a segment,
//     one to four waves per stream) covers the full row groups exactly once;
//   - plan_segments: batches of at most 64 segments, each below 2^31 chunks, every
//     non-empty segment exactly once and in order;
//   - grid_for stays below 2^32 work-items per dispatch; shapes are consistent;
//   - validation codes of check_params, check_segments, make_update_sweep, and the
//     coefficient function on edge inputs.
// Prints "plan_check ok" and returns 0, or names the first failed check and returns 1.

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <vector>

#include "zo.h"
#include "zo_plan.h"

using namespace zo;
typedef unsigned __int128 u128;

static int g_failed = 0;

#define CHECK(cond, ...)                                                       \
  do {                                                                         \
    if (!(cond)) {                                                             \
      if (g_failed++ < 20) {                                                   \
        std::fprintf(stderr, "FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond);   \
        std::fprintf(stderr, __VA_ARGS__);                                     \
        std::fprintf(stderr, "\n");                                            \
      }                                                                        \
    }                                                                          \
  } while (0)

// splitmix64: a seeded source of test cases
static uint64_t g_rng = 0x9E3779B97F4A7C15ull;
static uint64_t rnd() {
  uint64_t z = (g_rng += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// The kernels' walk over one plan's chunk slots (for_each_group): slot j of the segment holds
// groups [j cg - head, (j + 1) cg - head) clipped to [0, span), and only slots wholly before
// the first group (alignment slots) are empty; wave `sub` of a stream of `wps` waves takes
// every wps-th group of a slot. All of it in 32-bit arithmetic, as on the device; the 64-bit
// shadow checks that nothing wraps and that the groups are covered exactly once.
static void check_chunk_walk(const Plan& pl, uint32_t cg, uint32_t wps, const char* what) {
  const uint32_t chunks = plan_chunks(pl, cg);
  if (pl.span == 0) {
    CHECK(chunks == 0, "%s: chunks without full groups", what);
    return;
  }
  const u128 top64 = (u128)pl.head + pl.span;
  CHECK(top64 + cg < ((u128)1 << 32), "%s: slot arithmetic wraps", what);
  CHECK((u128)chunks * cg >= top64 && (u128)(chunks - 1) * cg < top64, "%s: chunk count", what);
  // every slot when few, else the leading ones, the first and last thousand and a sample
  std::vector<uint32_t> js;
  if (chunks <= 20000) {
    for (uint32_t j = 0; j < chunks; ++j) js.push_back(j);
  } else {
    for (uint32_t j = 0; j < 1000 + pl.head / cg; ++j) js.push_back(j);
    for (uint32_t j = chunks - 1000; j < chunks; ++j) js.push_back(j);
    for (int i = 0; i < 2000; ++i) js.push_back(static_cast<uint32_t>(rnd() % chunks));
  }
  uint64_t covered = 0;
  for (uint32_t j : js) {
    const u128 a64 = (u128)j * cg, b64 = a64 + cg;
    const u128 lo64 = a64 > pl.head ? a64 : (u128)pl.head, hi64 = b64 < top64 ? b64 : top64;
    // the device's 32-bit form
    const uint32_t a = j * cg, b = (j + 1) * cg, top = pl.head + pl.span;
    const uint32_t lo = a > pl.head ? a : pl.head, hi = b < top ? b : top;
    CHECK(lo == lo64 && hi == hi64, "%s: slot %u bounds", what, j);
    if (lo >= hi) {
      CHECK(b64 <= pl.head, "%s: slot %u empty after the first group", what, j);
      continue;
    }
    const uint32_t g0c = lo - pl.head, g1 = hi - pl.head;
    uint64_t in_chunk = 0;
    for (uint32_t sub = 0; sub < wps; ++sub) {
      if (lo + sub >= hi) continue;
      const uint32_t g0 = g0c + sub;
      const uint32_t cnt = (g1 - g0 + (wps - 1)) / wps;
      const uint64_t last = (uint64_t)g0 + (uint64_t)wps * (cnt - 1);
      CHECK(last < g1 && last + wps >= g1, "%s: wave %u of chunk %u", what, sub, j);
      in_chunk += cnt;
    }
    CHECK(in_chunk == (uint64_t)(g1 - g0c), "%s: chunk %u visits %llu of %u groups", what, j,
          (unsigned long long)in_chunk, g1 - g0c);
    covered += g1 - g0c;
  }
  if (chunks <= 20000) CHECK(covered == pl.span, "%s: chunks cover %llu of %u groups", what,
                             (unsigned long long)covered, pl.span);
}

// The memory chunk of a plan's slot j: slot boundaries sit at multiples of cg groups in memory.
static uint64_t mem_chunk_of(const Plan& pl, size_t elem, uint32_t cg, uint32_t j) {
  const uint64_t g_mem = reinterpret_cast<uintptr_t>(pl.gbase) / (kGroupElems * elem);  // memory group of group 0
  return (g_mem + (uint64_t)j * cg - pl.head) / cg;
}

// In a launch, every non-empty slot's launch chunk index is congruent to its memory chunk
// index modulo the streams of a workgroup, and slot boundaries sit at memory chunk boundaries
// (where the first full group sits at a group boundary in memory).
template <int N>
static void check_alignment(const Plans<N>& ps, size_t elem, uint32_t streams, const char* what) {
  const uint32_t cg = ps.chunk_groups;
  for (uint32_t s = 0; s < ps.count; ++s) {
    const Plan& pl = ps.p[s];
    if (!pl.span) continue;
    const uint32_t first = pl.head / cg, prev = s ? ps.chunk_end[s - 1] : 0;
    CHECK(pl.head < streams * cg, "%s: segment %u has %u alignment slots", what, s, first);
    const uint64_t g_mem = reinterpret_cast<uintptr_t>(pl.gbase) / (kGroupElems * elem);
    CHECK(pl.head % cg == g_mem % cg, "%s: segment %u slot boundaries", what, s);
    for (uint32_t j : {first, first + 1, ps.chunk_end[s] - prev - 1}) {
      if (prev + j >= ps.chunk_end[s]) continue;
      CHECK((prev + j) % streams == mem_chunk_of(pl, elem, cg, j) % streams,
            "%s: segment %u slot %u: launch chunk %u, memory chunk %llu", what, s, j, prev + j,
            (unsigned long long)mem_chunk_of(pl, elem, cg, j));
    }
  }
}

// make_plan's split of [offset, offset + n) into edge tiles and full row groups.
static void check_plan(uintptr_t addr, uint64_t offset, uint64_t n, size_t elem, uint32_t cg) {
  char what[160];
  std::snprintf(what, sizeof what, "plan(addr=%#llx, offset=%llu, n=%llu, elem=%zu, cg=%u)",
                (unsigned long long)addr, (unsigned long long)offset, (unsigned long long)n, elem, cg);
  const Plan pl = make_plan(reinterpret_cast<void*>(addr), offset, n, elem, cg);
  const u128 lo = offset, hi = (u128)offset + n;
  CHECK(pl.lo == offset && (u128)pl.hi == hi, "%s: range", what);
  const bool aligned = ((addr - (uintptr_t)(offset * elem)) & 15u) == 0;
  u128 head_end = hi, tail_begin = hi;
  if (pl.span) {
    CHECK(aligned, "%s: full groups on a misaligned base", what);
    const u128 f0 = (u128)pl.g_lo * kGroupElems, f1 = f0 + (u128)pl.span * kGroupElems;
    CHECK(f0 >= lo && f0 - lo < kGroupElems, "%s: first full group", what);
    CHECK(f1 <= hi && hi - f1 < kGroupElems, "%s: last full group", what);
    const uintptr_t gb = reinterpret_cast<uintptr_t>(pl.gbase);
    CHECK(pl.head == gb / (kGroupElems * elem) % cg, "%s: head", what);
    CHECK(gb == addr + (uintptr_t)((f0 - lo) * elem), "%s: gbase", what);
    CHECK((gb & 15u) == 0, "%s: gbase misaligned", what);
    head_end = f0;
    tail_begin = f1;
  } else if (aligned) {
    // no full group fits: [lo, hi) holds no multiple of 1024 followed by 1024 more elements
    const u128 f0 = (lo + kGroupElems - 1) / kGroupElems * kGroupElems;
    CHECK(f0 + kGroupElems > hi, "%s: a full group was left to the edge path", what);
  }
  // head tiles cover [lo, head_end), tail tiles [tail_begin, hi), one tile per 16 elements
  if (head_end > lo) {
    CHECK(pl.head_t0 == offset / kTile, "%s: head tile", what);
    const u128 t_end = ((u128)pl.head_t0 + pl.head_nt) * kTile;
    CHECK(pl.head_nt > 0 && t_end >= head_end && t_end - kTile < head_end, "%s: head tiles", what);
  } else {
    CHECK(pl.head_nt == 0, "%s: head tiles without a head", what);
  }
  if (hi > tail_begin) {
    CHECK((u128)pl.tail_t0 * kTile == tail_begin, "%s: tail tile", what);
    const u128 t_end = ((u128)pl.tail_t0 + pl.tail_nt) * kTile;
    CHECK(pl.tail_nt > 0 && t_end >= hi && t_end - kTile < hi, "%s: tail tiles", what);
  } else {
    CHECK(pl.tail_nt == 0, "%s: tail tiles without a tail", what);
  }
  if (aligned)  // storage misaligned relative to the global index takes the element path throughout
    CHECK((u128)pl.head_nt * kTile <= 2 * kGroupElems + kTile && (u128)pl.tail_nt * kTile <= kGroupElems + kTile,
          "%s: edge paths longer than a row group", what);
  for (uint32_t wps : {1u, 2u, 4u}) check_chunk_walk(pl, cg, wps, what);
}

// A tensor through plan_segments (one plan per launch, as zo_perturb launches one tensor):
// the plans' element ranges, in order, partition [offset, offset + n), each plan as check_plan
// requires, and every launch stays below 2^31 edge tiles.
static void check_pieces(uintptr_t addr, uint64_t offset, uint64_t n, size_t elem, uint32_t cg,
                         uint32_t streams = 4) {
  const zo_segment seg{reinterpret_cast<void*>(addr), offset, n};
  u128 next = offset;
  size_t plans = 0;
  const int rc = plan_segments<1>(&seg, 1, elem, cg, streams, [&](const Plans<1>& ps) {
    const Plan& pl = ps.p[0];
    check_alignment(ps, elem, streams, "pieces");
    if (pl.span) {
      for (uint32_t wps : {1u, 2u}) check_chunk_walk(pl, cg, wps, "launched piece");
    }
    CHECK(ps.count == 1 && pl.lo == next, "pieces out of order at %llu", (unsigned long long)pl.lo);
    CHECK((uint64_t)ps.edge_end[0] < kMaxLaunchEdges, "launch of %u edge tiles", ps.edge_end[0]);
    CHECK((u128)ps.edge_end[0] == (u128)pl.head_nt + pl.tail_nt, "edge count");
    const uintptr_t at = addr + (uintptr_t)((pl.lo - offset) * elem);
    CHECK(reinterpret_cast<uintptr_t>(pl.base) == at, "piece address");
    check_plan(at, pl.lo, pl.hi - pl.lo, elem, cg);
    next = (u128)pl.hi;
    ++plans;
    return static_cast<int>(ZO_OK);
  });
  CHECK(rc == ZO_OK && next == (u128)offset + n, "pieces cover up to %llu of %llu", (unsigned long long)(next - offset),
        (unsigned long long)n);
  if (groups_aligned(seg.params, offset, elem))
    CHECK(plans == 1, "an aligned tensor in %zu launches", plans);
  else
    CHECK(plans == (n + kPieceElems - 1) / kPieceElems, "%zu pieces", plans);
}

static void check_plans() {
  const uintptr_t A = 0x7f3200000000ull;  // a device-like address
  const uint64_t top = std::numeric_limits<uint64_t>::max();
  const uint64_t ns[] = {1, 15, 16, 17, 1000, 1023, 1024, 1025, 2047, 2048, 2049, 65549, 300000, (1ull << 20) + 3};
  const uint64_t offs[] = {0, 1, 7, 15, 16, 1023, 1024, 1025, (1ull << 32) - 1, (1ull << 35) + 7, 1ull << 60};
  for (size_t elem : {(size_t)2, (size_t)4})
    for (uint32_t cg : {1u, 2u, 4u, 8u, 16u})
      for (uint64_t n : ns)
        for (uint64_t off : offs)
          for (uintptr_t shift : {(uintptr_t)0, (uintptr_t)elem, (uintptr_t)8}) {
            check_plan(A + shift, off, n, elem, cg);
            // the buffer's first element at global index 2^64 - n - 1 .. 2^64 - n (top of the range)
            check_plan(A + shift, top - n, n, elem, cg);
            if (n > 1) check_plan(A + shift, top - n - off % 97, n, elem, cg);
          }
  // huge tensors: n up to ZO_N_MAX - 1 (2^30 row groups), at low and top offsets
  for (size_t elem : {(size_t)2, (size_t)4})
    for (uint32_t cg : {1u, 8u, 16u})
      for (uint64_t n : {ZO_N_MAX - 1, ZO_N_MAX - 1024, (1ull << 39) + 5, (1ull << 31) + 777})
        for (uint64_t off : {(uint64_t)0, (uint64_t)1023, (uint64_t)(1ull << 33) + 1, top - n, top - n - 5000}) {
          check_pieces(A, off, n, elem, cg, 16);
          check_pieces(A + elem, off, n, elem, cg);
        }
  // random cases
  for (int i = 0; i < 3000; ++i) {
    const size_t elem = rnd() & 1 ? 2 : 4;
    const uint32_t cg = 1u << (rnd() % 5);
    const uint64_t n = 1 + rnd() % (1ull << (rnd() % 24 + 1));
    uint64_t off = rnd() >> (rnd() % 64);
    if (off > top - n) off = top - n;
    // bases anywhere in a 128 KiB window, so that the alignment slots take every value
    const uint32_t streams = 1u << (rnd() % 5);
    check_pieces(A + (rnd() % 65536) * elem, off, n, elem, cg, streams);
  }
}

static void check_batches() {
  // 150 tensors of mixed sizes (and some empty ones) in one call
  std::vector<zo_segment> segs;
  uint64_t g = 0;
  for (int i = 0; i < 150; ++i) {
    const uint64_t n = i % 17 == 5 ? 0 : 1 + rnd() % 5000000;
    // most tensors 16-byte aligned relative to their global offset, at any 16-byte position
    // of a 128 KiB window (so the alignment slots take every value), some not aligned at all
    const uint64_t at = (i % 7 == 3 ? 2 : (2 * g) % 16) + 16 * (rnd() % 8192);
    segs.push_back({reinterpret_cast<void*>(0x7f0000000000ull + (uint64_t)i * (1ull << 26) + at), g, n});
    g += n + rnd() % 3;
  }
  CHECK(check_segments(segs.data(), (uint32_t)segs.size(), ZO_BF16) == ZO_OK, "disjoint segments rejected");
  std::vector<size_t> seen;
  size_t launches = 0;
  int rc = plan_segments<kSegsPerLaunch>(segs.data(), (uint32_t)segs.size(), 2, 16, 4, [&](const Plans<kSegsPerLaunch>& ps) {
    ++launches;
    CHECK(ps.count >= 1 && ps.count <= kSegsPerLaunch, "batch of %u segments", ps.count);
    check_alignment(ps, 2, 4, "batch");
    for (uint32_t s = 0; s < ps.count; ++s) {
      for (size_t i = 0; i < segs.size(); ++i)
        if (segs[i].params == ps.p[s].base && segs[i].n) seen.push_back(i);
      const uint32_t prev = s ? ps.chunk_end[s - 1] : 0;
      CHECK(ps.chunk_end[s] - prev == plan_chunks(ps.p[s], 16), "chunk count of segment %u", s);
      CHECK(ps.edge_end[s] - (s ? ps.edge_end[s - 1] : 0) == ps.p[s].head_nt + ps.p[s].tail_nt, "edge count");
    }
    return ZO_OK;
  });
  CHECK(rc == ZO_OK, "plan_segments status %d", rc);
  size_t nonempty = 0;
  for (auto& s : segs) nonempty += s.n != 0;
  CHECK(seen.size() == nonempty, "%zu of %zu segments launched", seen.size(), nonempty);
  for (size_t i = 1; i < seen.size(); ++i) CHECK(seen[i] > seen[i - 1], "segments out of order");
  CHECK(launches == (nonempty + kSegsPerLaunch - 1) / kSegsPerLaunch, "%zu launches", launches);

  // 40 tensors of ZO_N_MAX - 1 bf16 weights in 32 KiB chunks: 2^26 + 1 chunks each, so a launch
  // must close before 2^31 chunks
  std::vector<zo_segment> big;
  for (int i = 0; i < 40; ++i)
    big.push_back({reinterpret_cast<void*>((1ull << 44) + (uint64_t)i * (ZO_N_MAX * 2)), (uint64_t)i * ZO_N_MAX,
                   ZO_N_MAX - 1});
  CHECK(check_segments(big.data(), 40, ZO_BF16) == ZO_OK, "huge disjoint segments rejected");
  size_t total = 0;
  launches = 0;
  rc = plan_segments<kSegsPerLaunch>(big.data(), 40, 2, 16, 16, [&](const Plans<kSegsPerLaunch>& ps) {
    ++launches;
    CHECK((uint64_t)ps.chunk_end[ps.count - 1] < kMaxLaunchChunks, "launch of %u chunks", ps.chunk_end[ps.count - 1]);
    total += ps.count;
    return ZO_OK;
  });
  CHECK(rc == ZO_OK && total == 40 && launches == 2, "huge batches: %zu segments in %zu launches", total, launches);
  // a launch failure stops the batching with its status
  launches = 0;
  rc = plan_segments<kSegsPerLaunch>(segs.data(), (uint32_t)segs.size(), 2, 16, 4, [&](const Plans<kSegsPerLaunch>&) {
    ++launches;
    return ZO_ERR_HIP;
  });
  CHECK(rc == ZO_ERR_HIP && launches == 1, "failed launch not reported");
}

static void check_validation() {
  int dummy[4];
  void* p = dummy;
  const uint64_t top = std::numeric_limits<uint64_t>::max();
  CHECK(check_params(p, (zo_dtype)7, 0, 10) == ZO_ERR_ARG, "dtype");
  CHECK(check_params(nullptr, ZO_BF16, 0, 0) == ZO_OK, "empty");
  CHECK(check_params(nullptr, ZO_BF16, 0, 1) == ZO_ERR_NULL, "null");
  CHECK(check_params(reinterpret_cast<char*>(p) + 1, ZO_BF16, 0, 1) == ZO_ERR_ARG, "bf16 alignment");
  CHECK(check_params(reinterpret_cast<char*>(p) + 2, ZO_F32, 0, 1) == ZO_ERR_ARG, "f32 alignment");
  CHECK(check_params(p, ZO_F32, top - 10, 10) == ZO_OK, "top of the index range");
  CHECK(check_params(p, ZO_F32, top - 9, 10) == ZO_ERR_ARG, "index 2^64");
  CHECK(check_params(p, ZO_F32, top, top) == ZO_ERR_ARG, "wrapping range");
  CHECK(check_params(p, ZO_BF16, 0, ZO_N_MAX) == ZO_ERR_ARG, "n = ZO_N_MAX");
  CHECK(check_params(p, ZO_BF16, 0, ZO_N_MAX - 1) == ZO_OK, "n = ZO_N_MAX - 1");

  zo_segment ov[2] = {{reinterpret_cast<void*>(0x1000), 0, 100}, {reinterpret_cast<void*>(0x1000 + 198), 100, 10}};
  CHECK(check_segments(ov, 2, ZO_BF16) == ZO_ERR_ARG, "overlap");
  ov[1].params = reinterpret_cast<void*>(0x1000 + 200);
  CHECK(check_segments(ov, 2, ZO_BF16) == ZO_OK, "adjacent");
  ov[1].params = reinterpret_cast<void*>(UINTPTR_MAX - 7);
  CHECK(check_segments(ov, 2, ZO_BF16) == ZO_ERR_ARG, "segment past the end of the address space");
  CHECK(check_segments(nullptr, 3, ZO_BF16) == ZO_ERR_NULL, "null list");
  CHECK(check_segments(nullptr, 0, ZO_BF16) == ZO_OK, "empty list");

  std::vector<float> c(ZO_K_MAX + 1, 0.25f);
  Sweep w;
  CHECK(make_update_sweep(w, 0, ZO_K_MAX + 1, c.data(), 1e-3f, nullptr) == ZO_ERR_ARG, "K > K_MAX");
  CHECK(make_update_sweep(w, 0xFFFFFFC0u, 64, c.data(), 1e-3f, nullptr) == ZO_OK && w.n_groups == 8, "top probes");
  CHECK(make_update_sweep(w, 0xFFFFFFC1u, 64, c.data(), 1e-3f, nullptr) == ZO_ERR_ARG, "probe 2^32");
  CHECK(make_update_sweep(w, 3, 16, nullptr, 1e-3f, nullptr) == ZO_ERR_NULL, "null c");
  c[5] = std::numeric_limits<float>::quiet_NaN();
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, nullptr) == ZO_ERR_NONFINITE, "NaN c");
  c[5] = 0.25f;
  CHECK(make_update_sweep(w, 0, 16, c.data(), std::numeric_limits<float>::infinity(), nullptr) == ZO_ERR_NONFINITE,
        "inf lr");
  const Probe r0 = make_probe(15, 0.0f), r1 = make_probe(15, 1e-3f);
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, &r0) == ZO_OK && !w.restore, "zero restore");
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, &r1) == ZO_OK && w.restore && w.r.group == 1 && w.r.bit == 7,
        "restore probe");
  // the restore is merged into a table exactly when its probe group is one of the update's
  CHECK(w.fold, "restore of the last probe folds");
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, &r0) == ZO_OK && !w.fold, "zero restore does not fold");
  const Probe r_in = make_probe(3, 1e-3f), r_below = make_probe(7, 1e-3f), r_above = make_probe(40, 1e-3f);
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, &r_in) == ZO_OK && w.fold, "restore in the first group");
  CHECK(make_update_sweep(w, 8, 16, c.data(), 1e-3f, &r_below) == ZO_OK && w.restore && !w.fold,
        "restore below the update's groups");
  CHECK(make_update_sweep(w, 3, 13, c.data(), 1e-3f, &r1) == ZO_OK && w.fold, "restore in a partly used group");
  CHECK(make_update_sweep(w, 0, 16, c.data(), 1e-3f, &r_above) == ZO_OK && w.restore && !w.fold,
        "restore above the update's groups");
  const Probe r_top = make_probe(0xFFFFFFFFu, 1e-3f);
  CHECK(make_update_sweep(w, 0xFFFFFFC0u, 64, c.data(), 1e-3f, &r_top) == ZO_OK && w.fold, "restore of probe 2^32 - 1");
  CHECK(make_update_sweep(w, 0, 64, c.data(), 1e-3f, &r_top) == ZO_OK && !w.fold, "far restore does not fold");
  CHECK(make_update_sweep(w, 5, 1000, c.data(), 1e-3f, nullptr) == ZO_OK && w.n_groups == 126, "groups of 5..1004");
  const uint32_t kb = 9;
  const Sweep two = perturb_sweep(1, 1e-3f, &kb, -2e-3f);
  CHECK(two.two && two.b.group == 1 && two.b.bit == 1 && check_sweep(two) == ZO_OK, "two probes");
  const Sweep bad = perturb_sweep(1, std::numeric_limits<float>::infinity(), nullptr, 0.0f);
  CHECK(check_sweep(bad) == ZO_ERR_NONFINITE, "inf eps");
}

static void check_grids_and_shapes() {
  for (uint32_t block : {256u, 512u, 1024u})
    for (uint64_t items : {(uint64_t)1, (uint64_t)1000, (uint64_t)1 << 26, (uint64_t)1 << 31, (uint64_t)1 << 40})
      for (uint64_t per : {(uint64_t)1, (uint64_t)4, (uint64_t)16, (uint64_t)block})
        for (bool sized : {false, true}) {
          const uint32_t g = grid_for(items, per, block, sized);
          CHECK(g >= 1 && (uint64_t)g * block < (1ull << 32), "grid %u x %u", g, block);
          CHECK(sized || g <= kDefaultMaxBlocks, "unsized grid %u", g);
        }
  set_max_blocks(7);
  CHECK(grid_for(1ull << 30, 1, 256, true) == 7, "max blocks override");
  set_max_blocks(0xFFFFFFFFu);
  CHECK((uint64_t)grid_for(1ull << 40, 1, 1024, true) * 1024 < (1ull << 32), "override above the dispatch limit");
  set_max_blocks(0);
  std::vector<float> c(ZO_K_MAX, 0.5f);
  for (size_t elem : {(size_t)2, (size_t)4})
    for (uint64_t n : {(uint64_t)1000, (uint64_t)1 << 27, (uint64_t)12853473280ull})
      for (uint32_t K : {0u, 1u, 8u, 9u, 16u, 24u, 32u, 40u, 60u, 64u, 65u, 96u, 1024u})
        for (int kind = 0; kind < 4; ++kind) {
          Sweep w{};
          const uint32_t kb = 3;
          const Probe r = make_probe(K ? K - 1 : 0, 1e-3f);
          if (kind == 0) w = perturb_sweep(1, 1e-3f, nullptr, 0.0f);
          if (kind == 1) w = perturb_sweep(1, 1e-3f, &kb, 1e-3f);
          if (kind >= 2 && K && make_update_sweep(w, 0, K, c.data(), 1e-3f, kind == 3 ? &r : nullptr) != ZO_OK)
            CHECK(false, "update sweep K=%u", K);
          if (kind >= 2 && K == 0) continue;
          const Shape sh = shape_for(n, elem, w);
          CHECK(sh.chunk_groups >= 1 && sh.chunk_groups * kGroupElems * elem <= kMaxChunkBytes, "chunk");
          CHECK(sh.block % 64 == 0 && sh.block <= 1024 && sh.wps >= 1 && (sh.block / 64) % sh.wps == 0, "dims");
          CHECK(sh.copies == 0 || sh.copies == 16 || sh.copies == 32, "copies");
          CHECK(!w.update || sh.copies * w.n_groups <= 128, "tables beyond two planes");
          CHECK(occupancy_lds(sh.blocks_per_cu, 0) <= 96 * 1024, "occupancy pad");
        }
}

static void check_coefficients() {
  const uint32_t K = 1024;
  std::vector<double> lp(K), lm(K), c64(K), curv(K), w(K);
  std::vector<float> c(K);
  for (uint32_t k = 0; k < K; ++k) {
    lp[k] = 2.0 + (double)(rnd() % 1000) * 1e-4;
    lm[k] = 2.0 - (double)(rnd() % 1000) * 1e-4;
  }
  lp[1] = lm[1] = 2.0;  // zero curvature: w = 1
  lp[2] = 1e300;        // huge curvatures of either sign
  lm[3] = -1e300;
  CHECK(zo_probe_coeffs_ex(lp.data(), lm.data(), K, 2.0, 1e-3, 0.1, 1.0, c.data(), c64.data(), curv.data(), w.data()) ==
            ZO_OK, "coefficients");
  CHECK(w[1] == 1.0, "w at zero curvature");
  for (double a : {0.0, 0.1, 0.5, 1.0})
    CHECK(zo_probe_coeffs_ex(lp.data(), lm.data(), K, 2.0, 1e-200, a, 1.0, c.data(), nullptr, nullptr, nullptr) == ZO_OK,
          "eps^2 underflow, alpha %g", a);
  CHECK(zo_probe_coeffs_ex(lp.data(), lm.data(), K, 2.0, 1e-3, 1.5, 1.0, c.data(), nullptr, nullptr, nullptr) ==
            ZO_ERR_ARG, "alpha > 1");
  lp[7] = std::numeric_limits<double>::infinity();
  CHECK(zo_probe_coeffs(lp.data(), lm.data(), K, 2.0, 1e-3, c.data()) == ZO_ERR_NONFINITE, "inf loss");
  CHECK(zo_probe_coeffs(lp.data(), lm.data(), 0, 2.0, 1e-3, c.data()) == ZO_ERR_ARG, "K = 0");
  CHECK(zo_probe_coeffs(nullptr, lm.data(), 4, 2.0, 1e-3, c.data()) == ZO_ERR_NULL, "null losses");
  CHECK(zo_strerror(-99) != nullptr && zo_version() != nullptr, "strings");
}

int main() {
  check_validation();
  check_grids_and_shapes();
  check_plans();
  check_batches();
  check_coefficients();
  if (g_failed) {
    std::fprintf(stderr, "plan_check: %d checks failed\n", g_failed);
    return 1;
  }
  std::printf("plan_check ok\n");
  return 0;
}
