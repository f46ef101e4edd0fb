// Host-side launch planning of libzo's sweeps: argument validation, the split of a tensor
// into row groups, chunks and edge tiles, the launch shapes, and the batching of segment
// lists into launches. Plain C++ (no HIP), shared by the sweep launcher (zo_sweep.hip) and
// by the host checker that runs this code under AddressSanitizer and UBSan; the structs below
// are also the sweep kernels' arguments.
#ifndef ZO_PLAN_H_
#define ZO_PLAN_H_

#include <cstddef>
#include <cstdint>

#include "zo.h"

namespace zo {

constexpr uint32_t kTile = 16;              // elements per generator block
constexpr uint32_t kBlock = 256;            // threads per workgroup of the default launches (4 waves)
constexpr uint64_t kGroupElems = 1024;      // elements per row group (one Philox block per lane)
constexpr uint64_t kMaxChunkBytes = 32768;  // bytes a wave streams per chunk, at most
constexpr uint32_t kDefaultMaxBlocks = 65536;
constexpr uint32_t kSegsPerLaunch = 64;            // segments per batched launch (kernel arguments, ~5 KiB)
constexpr uint64_t kMaxLaunchChunks = 1ull << 31;  // chunks per launch: 32-bit indices with room for the stride
constexpr uint64_t kMaxLaunchEdges = 1ull << 31;   // edge tiles per launch, likewise
// Storage that is not 16-byte aligned relative to the global index has no full row groups:
// every element takes the element-wise path, one tile per lane. Such a tensor is planned in
// pieces of at most kPieceElems elements (2^30 tiles), so that edge-tile counts stay 32-bit.
constexpr uint64_t kPieceElems = 1ull << 34;
constexpr uint64_t kStreamBytes = 256ull << 20;    // sweeps at least this large stream (above the Infinity Cache)

// One segment: global elements [lo, hi) stored from `base` (the address of global element lo).
// The `span` full row groups from global group g_lo (stored from `gbase`) take the vector
// path, in chunk slots of `chunk_groups` groups whose boundaries sit at multiples of
// chunk_groups x the group's bytes in memory (as far as gbase's alignment allows): slot j
// holds the segment's groups [j chunk_groups - head, (j + 1) chunk_groups - head) clipped to
// [0, span). make_plan sets head = (gbase / group bytes) mod chunk_groups; add_plan adds whole
// empty slots in front (head grows by multiples of chunk_groups) so that a launch's chunk index
// and the memory index of the chunk agree modulo the streams of a workgroup, i.e. each
// workgroup streams one aligned block of memory (OPT-13B bf16 perturb: 7.65 ms with the
// workgroups' 128 KiB blocks aligned, 8.0-8.25 ms shifted by one to three 32 KiB chunks). The
// edge tiles [head_t0, +head_nt) and [tail_t0, +tail_nt) (fewer than 1024 elements at each
// end) take the element-wise path. The kernels walk chunks and groups with
// 32-bit indices relative to the segment (compares of 64-bit indices need a vector register
// on gfx950, and writing one that a pending store still reads makes the wave wait for that
// store); a segment stays below 2^30 row groups (n < ZO_N_MAX) and a launch below 2^31 chunks.
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

// One probe: bit `bit` of the probe bytes of generator group `group`, applied with weight eps.
struct Probe {
  uint32_t group, bit;
  float eps;
};

// The generator key (seed) and the step word of its counter.
struct Gen {
  uint32_t k0, k1, step;
};

struct Coefs {
  float c[ZO_K_MAX];
};

// What one sweep applies: one or two probes, or the update (with an optional restore probe).
// fold: the restore probe lies in one of the update's probe groups, so its +-eps is merged
// into that group's table and the sweep runs the plain update's per-element code.
struct Sweep {
  bool update;
  Probe a, b;
  bool two;
  uint32_t k_base, K, n_groups;
  Coefs cf;
  float lr;
  Probe r;
  bool restore;
  bool fold;
};

// The launch shape of a sweep.
struct Shape {
  uint32_t chunk_groups;
  uint32_t blocks_per_cu;    // 0: no cap
  uint32_t chunks_per_wave;  // 0: up to kDefaultMaxBlocks workgroups, grid-stride beyond
  uint32_t block = kBlock;   // threads per workgroup
  uint32_t wps = 1;          // waves per stream (per chunk)
  uint32_t copies = 0;       // update: copies of each table (0: one shared table)
};

// Whether global element 0 of a tensor stored from params with global offset `offset` would
// sit at a 16-byte boundary, which the full row groups need.
bool groups_aligned(const void* params, uint64_t offset, size_t elem);

// Validation (ZO_OK or the status the calls return; nothing is launched on an error).
int check_params(const void* params, zo_dtype dt, uint64_t offset, uint64_t n);
int check_segments(const zo_segment* segs, uint32_t n_segs, zo_dtype dtype);
int check_sweep(const Sweep& w);
int make_update_sweep(Sweep& w, uint32_t k_base, uint32_t K, const float* c, float lr, const Probe* r);
Sweep perturb_sweep(uint32_t k_a, float eps_a, const uint32_t* k_b, float eps_b);
Probe make_probe(uint32_t k, float eps);
Gen make_gen(uint64_t seed, uint32_t step);

// Planning.
Plan make_plan(void* params, uint64_t offset, uint64_t n, size_t elem, uint32_t chunk_groups);
uint32_t plan_chunks(const Plan& pl, uint32_t chunk_groups);
uint32_t grid_for(uint64_t work_items, uint64_t per_block, uint32_t block, bool sized = false);
Shape shape_for(uint64_t elements, size_t elem, const Sweep& w);
size_t occupancy_lds(uint32_t cap, size_t static_lds);
void set_max_blocks(uint32_t max_blocks);

// Streams (chunks in flight at once) of one workgroup of a launch shape.
inline uint32_t streams_per_block(const Shape& sh) { return sh.block / 64 / sh.wps; }

// Appends a plan to a launch: its chunk slots start at the launch's next chunk index after
// (memory chunk of its first full group - that index) mod `streams` empty slots, so that every
// chunk's launch index is congruent to its memory chunk index modulo `streams`.
template <int N>
void add_plan(Plans<N>& ps, Plan pl, size_t elem, uint32_t streams) {
  const uint32_t s = ps.count++;
  const uint32_t prev = s ? ps.chunk_end[s - 1] : 0;
  if (pl.span && streams > 1) {
    const uint64_t mem_chunk = reinterpret_cast<uintptr_t>(pl.gbase) / (kGroupElems * elem) / ps.chunk_groups;
    pl.head += static_cast<uint32_t>((mem_chunk % streams + streams - prev % streams) % streams) * ps.chunk_groups;
  }
  ps.p[s] = pl;
  ps.chunk_end[s] = prev + plan_chunks(pl, ps.chunk_groups);
  ps.edge_end[s] = (s ? ps.edge_end[s - 1] : 0) + pl.head_nt + pl.tail_nt;
}

// Workgroups of a launch: chunks_per_wave > 0, one workgroup per (streams per workgroup) x
// chunks_per_wave chunks; 0, up to kDefaultMaxBlocks workgroups, grid-stride beyond; and
// enough for the edge tiles, one per thread.
template <int N>
uint32_t plans_grid(const Plans<N>& ps, const Shape& sh) {
  const uint32_t chunks = ps.chunk_end[ps.count - 1], edges = ps.edge_end[ps.count - 1];
  const uint64_t streams = sh.block / 64 / sh.wps;
  const uint32_t cpw = sh.chunks_per_wave;
  const uint32_t a = chunks ? grid_for(chunks, streams * (cpw ? cpw : 1), sh.block, cpw > 0) : 1;
  const uint32_t b = grid_for(edges, sh.block, sh.block);
  return a > b ? a : b;
}

// A list of tensors in launches of up to N plans: calls launch(plans) for every batch.
// Segments with n = 0 are skipped; a segment without full row groups is planned in pieces of
// kPieceElems; a batch is closed before its chunk or edge-tile count would reach 2^31.
// `streams`: the streams of one workgroup of the launches (the chunk alignment of add_plan).
// Returns the first status launch() returns other than ZO_OK, else ZO_OK. The list must have
// passed check_segments.
template <int N, class Launch>
int plan_segments(const zo_segment* segs, uint32_t n_segs, size_t elem, uint32_t chunk_groups, uint32_t streams,
                  Launch launch) {
  Plans<N> ps{};
  ps.chunk_groups = chunk_groups;
  auto add = [&](const Plan& pl) {
    // the plan's chunks plus up to streams - 1 alignment slots
    if (ps.count && (ps.chunk_end[ps.count - 1] + static_cast<uint64_t>(plan_chunks(pl, chunk_groups)) + streams >=
                         kMaxLaunchChunks ||
                     ps.edge_end[ps.count - 1] + static_cast<uint64_t>(pl.head_nt) + pl.tail_nt >= kMaxLaunchEdges)) {
      const int rc = launch(ps);  // keep a launch's chunk and edge counts 32-bit
      if (rc != ZO_OK) return rc;
      ps.count = 0;
    }
    add_plan(ps, pl, elem, streams);
    if (ps.count == N) {
      const int rc = launch(ps);
      if (rc != ZO_OK) return rc;
      ps.count = 0;
    }
    return static_cast<int>(ZO_OK);
  };
  for (uint32_t i = 0; i < n_segs; ++i) {
    const zo_segment& sg = segs[i];
    const uint64_t piece = groups_aligned(sg.params, sg.offset, elem) ? sg.n : kPieceElems;
    for (uint64_t done = 0; done < sg.n; done += piece) {
      const uint64_t m = sg.n - done < piece ? sg.n - done : piece;
      void* at = reinterpret_cast<void*>(reinterpret_cast<uintptr_t>(sg.params) + static_cast<uintptr_t>(done * elem));
      const int rc = add(make_plan(at, sg.offset + done, m, elem, chunk_groups));
      if (rc != ZO_OK) return rc;
    }
  }
  return ps.count ? launch(ps) : ZO_OK;
}

}  // namespace zo

#endif  // ZO_PLAN_H_
