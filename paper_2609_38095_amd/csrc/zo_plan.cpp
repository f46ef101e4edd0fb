// Host-side launch planning of libzo's sweeps (declared in zo_plan.h): validation, the split
// of a tensor into row groups, chunks and edge tiles, and the launch shapes. Plain C++ with
// no HIP, compiled by the host compiler into libzo.so and, with AddressSanitizer and UBSan,
// into the host checker of the tests.

#include "zo_plan.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <utility>
#include <vector>

namespace zo {
namespace {

// zo_set_max_blocks: a cap on the workgroups of every later launch in the process (0: the
// default shapes). A test hook for grid independence; atomic so that a call on another thread
// sees either value, never a torn one.
std::atomic<uint32_t> g_max_blocks{0};

uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

}  // namespace

void set_max_blocks(uint32_t max_blocks) { g_max_blocks.store(max_blocks, std::memory_order_relaxed); }

// Workgroups for work_items items, per_block per workgroup of `block` threads, at most: the
// zo_set_max_blocks override if set, else kDefaultMaxBlocks, or (sized: the caller sized the
// work per workgroup itself) no cap; and always fewer than 2^32 work-items per dispatch. The
// kernels loop over whatever a smaller grid leaves.
uint32_t grid_for(uint64_t work_items, uint64_t per_block, uint32_t block, bool sized) {
  const uint64_t need = ceil_div(work_items, per_block);
  const uint32_t set = g_max_blocks.load(std::memory_order_relaxed);
  const uint64_t dispatch_cap = (1ull << 32) / block - 1;
  uint64_t cap = set ? set : sized ? dispatch_cap : kDefaultMaxBlocks;
  if (cap > dispatch_cap) cap = dispatch_cap;
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

// Full row groups need the address of global element 0 (params shifted back by offset
// elements; the subtraction may wrap, only its alignment is used) to be 16-byte aligned, so
// that every group vector is an aligned 16 bytes.
bool groups_aligned(const void* params, uint64_t offset, size_t elem) {
  return ((reinterpret_cast<uintptr_t>(params) - static_cast<uintptr_t>(offset * elem)) & 15u) == 0;
}

// The addresses are device addresses: they are only ever offset here, never dereferenced, and
// are carried as integers until the plan holds them. Without full row groups n must be at most
// kPieceElems (plan_segments splits larger tensors), so that the edge-tile counts fit 32 bits.
Plan make_plan(void* params, uint64_t offset, uint64_t n, size_t elem, uint32_t chunk_groups) {
  Plan pl{};
  pl.base = static_cast<char*>(params);
  pl.lo = offset;
  pl.hi = offset + n;
  if (n == 0) return pl;
  const uintptr_t addr = reinterpret_cast<uintptr_t>(params);
  uint64_t head_end = pl.hi, tail_begin = pl.hi;
  if (groups_aligned(params, offset, elem)) {
    const uint64_t g_lo = ceil_div(pl.lo, kGroupElems), g_hi = pl.hi / kGroupElems;
    if (g_lo < g_hi) {  // g_hi - g_lo < 2^30: n < ZO_N_MAX is checked first
      pl.g_lo = g_lo;
      pl.span = static_cast<uint32_t>(g_hi - g_lo);
      pl.gbase = reinterpret_cast<char*>(addr + static_cast<uintptr_t>((g_lo * kGroupElems - pl.lo) * elem));
      pl.head = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(pl.gbase) / (kGroupElems * elem) % chunk_groups);
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

// Chunk slots of a plan, the leading empty ones included (fewer than 2^30 + 2 + 16).
uint32_t plan_chunks(const Plan& pl, uint32_t chunk_groups) {
  return pl.span ? static_cast<uint32_t>(ceil_div(static_cast<uint64_t>(pl.head) + pl.span, chunk_groups)) : 0u;
}

Probe make_probe(uint32_t k, float eps) { return Probe{k / 8, k % 8, eps}; }

Gen make_gen(uint64_t seed, uint32_t step) {
  return Gen{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), step};
}

// Streaming shape of a launch over `elements` weights of `elem` bytes. HBM sustains these
// in-place sweeps best as few long sequential read-write streams: each stream walks up to
// kMaxChunkBytes of consecutive row groups with the next one or two groups in flight per wave,
// and occupancy is capped with dynamic LDS so that few streams run at once (the bf16 perturb
// on an OPT-13B shaped buffer: 6.5 TB/s at one workgroup per CU, 5.6 at full occupancy). An
// update needs more waves where its generator and table work per byte outgrows what one wave
// overlaps with its own loads: either two waves per stream (each takes every other row group
// of the chunk, so the stream keeps its length and gains a second wave to hide the work) or
// larger workgroups that share one set of spread tables. The shapes below are the fastest of
// those measured (A/B on one box) on OPT-13B shaped bf16 buffers (K <= 16), OPT-30B (K = 32),
// OPT-1.3B and Qwen3-8B (K = 60-64) and 3 G-element fp32 buffers:
//   perturb, one or two probes: 256 threads, one workgroup per CU;
//   update, one bf16 group: one workgroup per CU, one chunk per wave (OPT-30B K = 8: 6.19 ->
//     6.53 TB/s), paced at four outstanding memory operations as the perturb (+0.5%);
//   update, two bf16 groups: 512 threads, two waves per stream, one chunk per stream, 32-copy
//     tables (OPT-13B K = 16: +0.5 to 1.8%, +2% on a GPU already busy with perturbs), paced
//     at four outstanding memory operations (+0.3 to 0.5% on three boxes; 2, 3, 5, 6 and 8,
//     three groups in flight, 16-copy tables, 256 threads and one wave per stream all equal
//     or slower);
//   update, three bf16 groups: three workgroups per CU, one group ahead;
//   update, four bf16 groups: 1024 threads, 32-copy tables in two planes (OPT-30B K = 32:
//     21.9 -> 21.6 ms);
//   update, eight bf16 groups (K = 57-64): 1024 threads sharing 16-copy tables in two planes
//     (4 LDS cycles per 64-lane read instead of 6.3), four chunks per stream (OPT-1.3B K = 64:
//     1.80 -> 1.57 ms; Qwen3-8B K = 60: 10.9 -> 9.9 ms);
//   fp32 updates: one workgroup per CU up to three groups, two at four, three at five or six.
// An update with a restore probe inside its groups (Algorithm 1's schedule) is the plain
// update with that group's table changed, and takes the update's shape. Other updates (five to
// seven bf16 groups, more than eight, or more than six in fp32, and a restore probe outside
// the update's groups) are bound by the generator or the LDS table lookups and keep 4 KiB
// chunks at full occupancy, as do perturbs smaller than the 256 MiB Infinity Cache (updates
// of such buffers take 8 KiB chunks at full occupancy). Grids: up to
// kDefaultMaxBlocks workgroups, grid-stride beyond (in-order dispatch of many short-lived
// workgroups keeps the streams compact; a persistent grid of one workgroup per CU measured
// 5.6 TB/s), except where a number of chunks per stream is given: the bf16 perturb of one
// probe or of two in one probe group, the two-probe fp32 perturb and the bf16 updates of one
// or two groups run one chunk per stream (OPT-13B: the perturb 6.48 -> 6.67 TB/s, OPT-30B
// 6.20 -> 6.60; two probes in one group +1%, across two groups -0.3%, so those stay
// grid-stride; 3 G fp32 weights: the two-probe perturb 6.30 -> 6.48 across two probe groups).
Shape shape_for(uint64_t elements, size_t elem, const Sweep& w) {
  const uint64_t group_bytes = kGroupElems * elem;
  const Shape short_chunks{static_cast<uint32_t>(4096 / group_bytes ? 4096 / group_bytes : 1), 0, 0};
  if (elements * elem < kStreamBytes) {
    if (!w.update) return short_chunks;
    // updates of cache-sized buffers: 8 KiB chunks, so that each workgroup's table build
    // serves twice the bytes (OPT-125M: K = 16 0.088 -> 0.084 ms, K = 60 0.201 -> 0.189 ms;
    // 16 and 32 KiB chunks measured slower at K = 16)
    return Shape{static_cast<uint32_t>(8192 / group_bytes), 0, 0};
  }
  const uint32_t chunk = static_cast<uint32_t>(kMaxChunkBytes / group_bytes);
  if (!w.update) {
    // one chunk per wave: bf16 with one probe or two in one group, fp32 with two probes
    const bool one_group_bf16 = elem == 2 && (!w.two || w.a.group == w.b.group);
    const bool two_probes_fp32 = w.two && elem == 4;
    return Shape{chunk, 1, one_group_bf16 || two_probes_fp32 ? 1u : 0u};
  }
  if (w.restore && !w.fold) return short_chunks;
  const uint32_t g = w.n_groups;
  Shape sh{chunk, 1, 0};
  if (elem == 4) {
    sh.blocks_per_cu = g <= 3 ? 1 : g == 4 ? 2 : g <= 6 ? 3 : 0;
    if (sh.blocks_per_cu == 0) return short_chunks;
    if (g <= 2) sh.copies = 32;  // one or two fp32 groups: 32-copy tables, one workgroup per CU
    return sh;
  }
  switch (g) {
    case 1:
      sh.chunks_per_wave = 1;  // one shared table: a single group leaves the LDS half idle
      return sh;
    case 2:
      sh.copies = 32;
      sh.wps = 2;
      sh.chunks_per_wave = 1;
      sh.block = 512;
      return sh;
    case 3:
      sh.blocks_per_cu = 3;
      return sh;
    case 4:
      sh.block = 1024;
      sh.copies = 32;
      return sh;
    case 8:
      sh.copies = 16;
      sh.block = 1024;
      sh.chunks_per_wave = 4;
      return sh;
    default:
      return short_chunks;
  }
}

// Dynamic LDS that, with `static_lds` bytes of the kernel's own, admits exactly `cap`
// workgroups on a CU's 160 KiB (0: no cap).
size_t occupancy_lds(uint32_t cap, size_t static_lds) {
  if (cap == 0) return 0;
  const size_t per_block = cap == 1 ? 96 * 1024 : cap == 2 ? 72 * 1024 : cap == 3 ? 48 * 1024 : 36 * 1024;
  return per_block > static_lds ? per_block - static_lds : 0;
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
  w.fold = w.restore && r->group - g_first < w.n_groups;  // wraps for a group below g_first
  return ZO_OK;
}


// A list of tensors is validated as a whole: alignment, index ranges, and no two segments
// sharing memory.
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

Sweep perturb_sweep(uint32_t k_a, float eps_a, const uint32_t* k_b, float eps_b) {
  Sweep w{};
  w.a = make_probe(k_a, eps_a);
  w.two = k_b != nullptr;
  w.b = k_b ? make_probe(*k_b, eps_b) : w.a;
  return w;
}

}  // namespace zo
