// Device-side data layout shared by the host part (space build) and the kernels of libmist.
#pragma once

#include <stdint.h>

#include "mist.h"

namespace mist {

constexpr int kBlock = 256;           // threads per evaluation block
constexpr int kWaves = kBlock / 64;   // wave64
constexpr int kWaveTile = 64;         // threads per tile: each wave works on its own tiles
constexpr int kReduceBlock = 256;     // filter block: one wave per group
constexpr int kTabStride = 8;         // interference table row: phi[4], psi[4]
constexpr int kClaimCounters = 8;     // tile counters: one per XCD (blocks are dealt in turn)
constexpr int kCounterStride = 64;    // ints between counters (separate cache lines)
constexpr int kMaxAlphas = 16;        // weight samples of the (t, d) frontier

// One candidate stage (group): hardware sample, G, PP, in-flight count k, layers l.
struct DevGroup {
  uint64_t base;        // global id of the first configuration
  int32_t hw;
  int32_t G, PP, k, l;
  int32_t pair_begin;   // first (b, TP) pair in the pair table
  int32_t n_pairs;
  int32_t tile_begin;   // first of the group's full-size tiles in the tile table
  int32_t n_tiles;
  int32_t pk_begin;     // first entry of the group's pairs in the pair-constant table
  int32_t tail_begin;   // first of the group's small tiles (after every group's full-size ones)
  int32_t n_tail;
};

// One (b, TP) pair of a group, DP = D / (PP * TP).
struct DevPair {
  int32_t b, tp, dp, mb;  // mb: index of b in the microbatch list
  double inv_dp;          // 1 / DP, host division
};

// A wave's work item: strips [strip_begin, strip_end) of one group.  A strip is one
// (pair, recomputed layers, ZeRO level, weight ratio, gradient ratio) combination and
// holds the R^2 configurations of its (optimizer ratio, activation ratio) digits; strip s
// of a group covers local ids [s * R^2, (s + 1) * R^2).
struct DevTile {
  int32_t group;
  int32_t strip_begin;
  int32_t strip_end;
  int32_t pad;
};

// Per hardware sample: host reciprocals, bucket edges and the interference table.
struct DevHw {
  double iF, iP, iL;         // 1 / FLOP/s, 1 / PCIe, 1 / link
  double M;                  // memory budget
  double kNB;                // NB / M * (1 - 2^-40): floor(mem * kNB) is the bucket or one below
  double ieta[MIST_MAX_MB];  // 1 / eta(b) per microbatch index
  double edge[MIST_MAX_BUCKETS];     // E_j; +inf past NB
  // Row per co-running pattern (bit j = stream j runs): phi[4] then psi[4].  Patterns of
  // two or more streams: members carry phi and psi = 1/phi, other streams phi = +inf and
  // psi = 1 (their 0 or NaN time scales to NaN, which min/max skip).  Patterns of at most
  // one stream: phi = psi = 1 everywhere (no update).
  double itab[16][kTabStride];
};

struct DevModel {
  int64_t h, heads, kv, f, s, V, bw, bo;
  int32_t gpt, flash;
};

// Pair-level constants of one (group, pair): the cost-model quantities that depend on
// the stage and on (b, TP, DP) only (written by the pair kernel, read per strip).
struct PairK {
  int64_t afull, ack;  // activation bytes of a stored / checkpointed layer
  double Pw, Po;       // stage parameter bytes: fp16 copy, optimizer states
  double Wb2, Ob2o;    // double-buffered per-layer units: fp16, optimizer states
  double A2, AF, Xd;   // 2 x layer activations, layer activations, fp32 logits
  double Fld, Fh3;     // layer forward FLOPs, 3 x LM-head forward FLOPs
  double r, p2p, ar;   // seconds: one ZeRO AG/RS, pipeline sends, one TP all-reduce
  double FE;           // 1 / (F * eta(b))
  double iD;           // 1 / DP
};

// Candidate filter of the exact frontier, per (group, bucket j): the objective below which a
// configuration of bucket j can beat every lower bucket (exclusive prefix minimum of the bucket
// minima), and the objective and memory of bucket j's winner.
struct FiltEntry {
  double pm, bobj, bmem;
};

// Evaluation kernel variants.
constexpr int kModeBuckets = 0;  // bucket minima (and per-tile partials)
constexpr int kModeAlpha = 1;    // bucket minima and the weight-sampled argmins
constexpr int kModeEmit = 2;     // exact frontier: write and count each tile's candidates
constexpr int kModeDump = 3;     // per-configuration values of listed tiles (parity checks)
constexpr int kDumpWords = 6;    // doubles per configuration in the dump variant's output

struct EvalArgs {
  DevModel m;
  const DevGroup* groups;
  const DevPair* pairs;
  const DevTile* tiles;
  const int32_t* tile_order;  // [n_tiles] work item -> tile of the persistent grid (nullptr:
                              // item x is tile x)
  const DevHw* hws;
  const double* ratio;   // r[0..R), then om[0..R) = 1 - r
  int32_t R, NB;
  int32_t n_tiles;
  int32_t* work;         // tile counters of the persistent evaluation kernel, kClaimCounters
                         // of them kCounterStride apart (reset by K0)
  int64_t n_groups;
  uint64_t n_configs;
  double* part_obj;      // [n_tiles][64]
  uint64_t* part_id;     // [n_tiles][64]
  PairK* pk;             // [n_pk] pair constants, group-major
  const int32_t* pk_group;  // [n_pk] group of each entry
  int32_t n_pk;
  // Weight samples of Eq. 4 (n_alpha = 0: off): alpha[a] and 1 - alpha[a], and the per-tile
  // argmin of fma(alpha*G, t, (1-alpha)*d) over feasible configurations.
  int32_t n_alpha;
  const double* alpha;   // [n_alpha]
  const double* beta;    // [n_alpha]
  double* part_aobj;     // [n_tiles][n_alpha]
  uint64_t* part_aid;    // [n_tiles][n_alpha]
  // Exact frontier (emit variant).  Tile t writes its candidates, in evaluation order, to
  // slots [win_begin[t], win_end[t]) of cand_* and drops those past the window; its total
  // count goes to cnt_tile[t].  With tile_list set, the kernel runs only the n_list tiles
  // listed there.
  const FiltEntry* filt;     // [n_groups][64]
  int32_t* cnt_tile;         // [n_tiles]
  const int64_t* win_begin;  // [n_tiles]
  const int64_t* win_end;    // [n_tiles]
  const int32_t* tile_list;  // nullptr: every tile
  int32_t n_list;
  const uint8_t* tile_live;  // nullptr, or 0 for a tile that holds no candidate (skipped)
  uint64_t* cand_key;        // memory bit patterns (a non-negative double orders like its bits)
  double* cand_obj;
  uint64_t* cand_id;
  // Overflow pool of the first candidate pass (pool_count = nullptr: none).  A candidate past its
  // tile's window takes the next pool slot from *pool_count (reset by the pair kernel) and
  // stores itself with its tile and its rank among the tile's candidates; past pool_cap it is
  // dropped and tile_drop[t] = 1 marks the tile for a second evaluation.
  unsigned long long* pool_count;
  int64_t pool_cap;
  uint64_t* pool_key;
  double* pool_obj;
  uint64_t* pool_id;
  int32_t* pool_tile;
  int32_t* pool_rank;
  uint8_t* tile_drop;        // [n_tiles]
  // Dump variant (parity checks): listed item x writes, for every configuration of its tile in
  // local-id order, t, d, mem, obj, the bucket entry the kernel chose (as a double; NB..64 are
  // the sinks of infeasible configurations) and the forms of interference the kernel took
  // (first microbatch + 8 x stable time, as a double) to dump[kDumpWords * (dump_off[x] + i)..].
  double* dump;
  const int64_t* dump_off;   // [n_list]
};

struct ReduceArgs {
  const DevGroup* groups;
  int64_t n_groups;
  int32_t NB;
  int32_t max_group_tiles;  // tiles of the largest group (chooses the reduction's layout)
  const double* part_obj;
  const uint64_t* part_id;
  double* bucket_obj;    // [n_groups][64]
  uint64_t* bucket_id;   // [n_groups][64]
  double* best_obj;      // [n_groups]
  uint64_t* best_id;     // [n_groups]
  uint64_t* frontier;    // [n_groups]
  int32_t n_alpha;
  const double* part_aobj;
  const uint64_t* part_aid;
  double* alpha_obj;     // [n_groups][n_alpha]
  uint64_t* alpha_id;    // [n_groups][n_alpha]
};

// Allocation-free per-id evaluation (mist_eval_ids_noalloc): a fixed device scratch array of
// this many bytes holds the ids and the results of one call (40 bytes per id).
constexpr size_t kNoAllocScratchBytes = (size_t)4 << 20;
constexpr int64_t kNoAllocMaxIds = (int64_t)(kNoAllocScratchBytes / (sizeof(uint64_t) + 4 * sizeof(double)));
// The current device's address of that array (mist_noalloc.hip); 0 or a hipError_t.
int noalloc_scratch(void** ptr);

// Kernel launchers (mist_kernels.hip).
int launch_pairs(const EvalArgs& a, void* stream);
int launch_eval(const EvalArgs& a, int blocks, int mode, void* stream);
int eval_blocks_per_cu(int R, int mode);
int launch_reduce(const ReduceArgs& a, void* stream);
int launch_eval_ids(const EvalArgs& a, const uint64_t* ids, int64_t n, double* out, void* stream);
// Tiles that may hold a candidate of the exact frontier, from the last evaluation's partials.
int launch_live(const EvalArgs& a, const FiltEntry* filt, uint8_t* live, void* stream);
int launch_filter(const EvalArgs& a, const double* bucket_obj, const uint64_t* bucket_id, FiltEntry* filt,
                  void* stream);
// Exact frontier, mist_exact.hip: the candidates of group g are [seg[g], seg[g+1]).  The
// pre-filter drops, per group, candidates that one of strictly smaller memory dominates and
// moves the rest to the front (their end in seg_end); one segmented sort by memory over
// [seg[g], seg_end[g]) leaves the sorted keys in key_out and the candidates' slots in idx_out
// (key_tmp, idx_tmp: scratch of the same slots for large groups), and the per-group scan keeps
// the staircase.
int launch_prefilter(uint64_t* cand_key, double* cand_obj, uint64_t* cand_id, const int64_t* seg,
                     int64_t n_groups, int64_t* seg_end, void* stream);
int exact_sort(const uint64_t* cand_key, uint64_t* key_out, uint32_t* idx_out, uint64_t* key_tmp, uint32_t* idx_tmp,
               int64_t n_groups, const int64_t* seg_begin, const int64_t* seg_end, void* stream);
// Moves each tile's window [slab_begin[t], slab_begin[t+1]) (its first candidates, at most
// cnt[t]) to [tile_off[t], ...); tiles with tile_drop[t] set are skipped (evaluated again).
int launch_compact(const uint64_t* slab_key, const double* slab_obj, const uint64_t* slab_id,
                   const int64_t* slab_begin, const int32_t* cnt, const uint8_t* tile_drop, const int64_t* tile_off,
                   int32_t n_tiles, uint64_t* cand_key, double* cand_obj, uint64_t* cand_id, void* stream);
// Moves pool slots [0, n) to tile_off[pool_tile] + pool_rank (tiles with tile_drop set skipped).
int launch_pool_place(const uint64_t* pool_key, const double* pool_obj, const uint64_t* pool_id,
                      const int32_t* pool_tile, const int32_t* pool_rank, int64_t n, const uint8_t* tile_drop,
                      const int64_t* tile_off, uint64_t* cand_key, double* cand_obj, uint64_t* cand_id,
                      void* stream);
int launch_front_scan(const uint32_t* order, const uint64_t* sorted_key, const double* cand_obj,
                      const uint64_t* cand_id, const int64_t* seg_begin, const int64_t* seg_end, int64_t n_groups,
                      uint64_t* front_key, double* front_obj, uint64_t* front_id, int64_t* front_cnt, void* stream);

}  // namespace mist
