/*
 * libmist — batched evaluation of Mist's intra-stage tuner on one MI355X (gfx950).
 *
 * Zhu et al., "Mist: Efficient Distributed Training of Large Language Models via
 * Memory-Parallelism Co-Optimization", EuroSys '25.
 *
 * Problem (Sec. 5.3): given a model, a global batch B and a device mesh, intra-stage
 * tuning scores every per-stage tuple of Table 2 — microbatch b, DP, TP, ZeRO level,
 * recomputed layers, and the weight / gradient / optimizer-state / activation offload
 * ratios — for every candidate stage, by its peak memory (the constraint of Eq. 4) and its
 * stable-microbatch time t and first-microbatch delta d (Eq. 5-6) from the interference
 * model (Algorithm 1, Sec. 5.2.2); it keeps the feasible minimum of G*t + d per stage and a
 * time-versus-memory staircase over 64 memory buckets, which the inter-stage partitioner
 * (Eq. 1-3) consumes.
 *
 * A "group" is one candidate stage: (hardware sample, G, PP, k, l) with k the 1F1B
 * in-flight count of the stage position (k = PP first stage, 1 last) and l its layers.
 * Groups are numbered in ascending order of hw, PP, G, k, l.  Within a group a
 * configuration has the canonical local id
 *     ((((((p*(l+1) + c)*4 + z)*R + wo)*R + go)*R + oo)*R + ao)
 * with p the index of (b, TP) among the group's pairs in ascending order, c the recomputed
 * layers, z the ZeRO level and wo, go, oo, ao indices into the ratio list of length R;
 * its global id is the group's base plus the local id.
 *
 * Conventions
 *  - Every entry point returns a mist_status; nothing aborts and no C++ exception crosses
 *    the ABI.  On failure mist_last_error() returns a message (thread-local, valid until
 *    the next call on the same thread).
 *  - One mist_space must not be used from two threads at once; distinct spaces are
 *    independent.
 *  - Pointers named "host" are host memory owned by the caller.  Device memory is owned by
 *    the space and released by mist_space_destroy.
 */
#ifndef MIST_H
#define MIST_H

#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t mist_status;
#define MIST_OK 0
#define MIST_E_INVALID (-1) /* bad descriptor or argument */
#define MIST_E_NOMEM (-2)   /* host or device allocation failed */
#define MIST_E_DEVICE (-3)  /* a HIP call failed; the message carries hipGetErrorString */
#define MIST_E_STATE (-4)   /* results requested before mist_eval_space */
#define MIST_E_RANGE (-5)   /* index out of range or output capacity too small */

#define MIST_ARCH_GPT 0   /* LayerNorm, GeLU MLP of width ffn, learned positions */
#define MIST_ARCH_LLAMA 1 /* RMSNorm, SwiGLU MLP of width ffn, grouped-query attention */

#define MIST_L_FULL 0     /* stage layer counts 1..L-PP+1 (PP = 1: L) */
#define MIST_L_BALANCED 1 /* stage layer counts floor(L/PP) and ceil(L/PP) */

#define MIST_MAX_BUCKETS 64
#define MIST_MAX_ALPHAS 16
#define MIST_MAX_STAGES 64
#define MIST_MAX_RATIOS 16
#define MIST_MAX_MB 16
#define MIST_NONE UINT64_MAX /* id of an empty bucket or of a group with no feasible config */

/* Model shape (Sec. 6.1, Table 4; the transformer of the symbolic trace, Sec. 5.2.1). */
typedef struct mist_model_desc {
  int32_t arch;      /* MIST_ARCH_GPT or MIST_ARCH_LLAMA */
  int32_t n_layers;  /* L */
  int64_t hidden;    /* h; divisible by heads */
  int32_t heads;     /* attention heads */
  int32_t kv_heads;  /* key/value heads; divides heads */
  int64_t ffn;       /* MLP width f */
  int64_t seq;       /* sequence length s */
  int64_t vocab;     /* V */
  int32_t bytes_w;   /* bytes per fp16/bf16 weight, gradient and activation element (2) */
  int32_t bytes_opt; /* optimizer bytes per parameter: fp32 master + Adam m, v (12) */
  int32_t flash;     /* 1: FlashAttention, no stored attention probabilities */
} mist_model_desc;

/* One hardware sample: the inputs of the runtime model (Sec. 5.2.1: compute from the
 * operator database, communication as bytes / bandwidth) and of the interference model
 * (Sec. 5.2.2: one slowdown factor per co-running combination and stream). */
typedef struct mist_hw_desc {
  double flops;      /* peak FLOP/s, in [2^-200, 2^200] */
  double mem_bytes;  /* memory budget in bytes, > 0 (the Mem_Budget of Eq. 4) */
  double pcie_bw;    /* host<->device bytes/s, in [2^-200, 2^200] */
  double link_bw;    /* device<->device bytes/s, in [2^-200, 2^200] */
  double eta_max;    /* compute efficiency eta(b) = eta_max*b*s/(b*s + n_half), in [2^-100,
                        2^100]; 0 selects eta_tab */
  double n_half;     /* in [0, 2^100] */
  double phi[16][4]; /* phi[mask][j]: slowdown of stream j (0 compute, 1 GPU-GPU, 2 host->
                        device, 3 device->host) when the streams of mask co-run; in [1, 2^100];
                        entries of absent streams and single-stream masks unused */
  double eta_tab[MIST_MAX_MB]; /* with eta_max = 0: measured efficiency of the space's i-th
                        microbatch size, in [2^-100, 2^100], e.g. from mist_measure_eta (the
                        operator database of Sec. 5.2.1); unused otherwise */
} mist_hw_desc;
/* The magnitude bounds lie far beyond any physical value; they keep every non-zero stream time
 * of the runtime model within [2^-363, 2^500], so that no step of Algorithm 1 underflows. */

/* The search space of Table 2 for every candidate stage. */
typedef struct mist_space_desc {
  int64_t n_devices;     /* D */
  int64_t global_batch;  /* B */
  const int32_t* mb;     /* host: microbatch sizes, strictly ascending, >= 1 */
  int32_t n_mb;          /* 1..MIST_MAX_MB */
  const double* ratios;  /* host: offload ratios, strictly ascending in [0, 1]; a non-zero ratio
                            is at least 2^-100 */
  int32_t n_ratios;      /* R, 1..MIST_MAX_RATIOS */
  int32_t n_buckets;     /* NB, 1..MIST_MAX_BUCKETS; bucket edges E_j = M*(j+1)/NB */
  int32_t l_rule;        /* MIST_L_FULL or MIST_L_BALANCED */
  int32_t n_alphas;      /* 0..MIST_MAX_ALPHAS weight samples of Eq. 4; 0 (or a zeroed tail of
                            the struct) turns the weight-sampled argmins off */
  const double* alphas;  /* host: the samples alpha_a in [0, 1] (any order, repeats allowed) */
  int64_t tile_configs;  /* launch geometry, results do not depend on it: configurations per
                            full-size tile of the evaluation kernel, at least (0: 16384) */
  int32_t max_blocks;    /* cap on the evaluation kernel's grid (0: every block that fits on the
                            device at once) */
  int32_t cand_window;   /* exact frontier, results do not depend on it: each tile first writes
                            its candidates to a window of ceil(configurations / cand_window)
                            slots (0: 8, raised as needed to keep all windows within 2^27 slots),
                            the rest to an overflow pool of as many slots as all windows (at
                            most 2^27); a tile with a candidate that finds no place is
                            evaluated a second time */
} mist_space_desc;

/* Device memory provider, e.g. PyTorch's caching allocator.  alloc returns NULL on
 * failure; free receives exactly the pointers alloc returned.  hip_stream (a hipStream_t) is
 * the stream on which the library first uses the block, so that a stream-ordered allocator can
 * hand out a block whose earlier users were on that same stream: the null stream for the
 * space's own buffers (mist_space_create waits for the null stream before it returns, and later
 * calls may use them on any stream), the call's stream for the exact frontier's buffers and
 * for temporaries.  The library frees a block only after its own work on it has finished. */
typedef struct mist_allocator {
  void* (*alloc)(size_t bytes, void* hip_stream, void* ctx);
  void (*free)(void* ptr, void* ctx);
  void* ctx;
} mist_allocator;

typedef struct mist_space mist_space;

/* A decoded configuration (the per-stage tuple of Table 2 plus its group key). */
typedef struct mist_config {
  int32_t hw, G, PP, k, l;       /* group key */
  int32_t b, tp, dp, zero, ckpt; /* microbatch, TP, DP, ZeRO level 0..3, recomputed layers */
  int32_t wo_idx, go_idx, oo_idx, ao_idx; /* indices into the ratio list */
  double wo, go, oo, ao;         /* the ratios */
} mist_config;

typedef struct mist_result {
  uint64_t id;    /* MIST_NONE when no feasible configuration */
  double obj;     /* G*t + d; +inf when none */
  double t;       /* stable-microbatch time (s), Eq. 5 */
  double d;       /* first-microbatch delta (s), Eq. 6 */
  double mem;     /* max(forward peak, backward peak) in bytes, Eq. 4 */
  int32_t bucket; /* memory bucket of mem; -1 when none */
  int32_t pad;
  mist_config cfg;
} mist_result;

/* One intra-stage candidate for the inter-stage planner: a configuration of group
 * (G, PP, k, l) of one hardware sample with its stable time t and first-microbatch delta d
 * (seconds). */
typedef struct mist_stage_point {
  int32_t G, PP, k, l;
  uint64_t id;
  double t, d;
} mist_stage_point;

typedef struct mist_stage_plan {
  int32_t l, k;   /* layers of the stage; microbatches in flight (PP - i + 1 for stage i) */
  uint64_t id;    /* the stage's configuration */
  double t, d;
} mist_stage_plan;

/* A pipeline plan (Sec. 5.3, Eq. 1-3) for one hardware sample. */
typedef struct mist_plan {
  int32_t found;  /* 0 when no plan exists (then F = +inf) */
  int32_t hw, G, PP;
  double F;       /* Eq. 2: (G-1)*max t_i + sum t_i + max_i (d_i - sum_{j<i} t_j), in stage order */
  mist_stage_plan stage[MIST_MAX_STAGES];  /* stages 1..PP */
} mist_plan;

typedef struct mist_group_key {
  int32_t hw, G, PP, k, l, n_pairs;
  uint64_t base;  /* id of the group's first configuration */
  uint64_t size;  /* configurations in the group */
} mist_group_key;

/* The problem statement of Sec. 5.3: a model (m), hardware samples (hw) and a search space (s)
 * of the per-stage tuples of Table 2.  Validates and copies the descriptors (the caller may
 * free them afterwards), enumerates the groups (every candidate stage, the IntraStagePareto
 * queries of Eq. 3), builds the tables and uploads them to the current HIP device.  hw points
 * to n_hw >= 1 samples.  alloc may be NULL (hipMalloc/hipFree).  On success *out owns every
 * device and host buffer.  A space may hold no configuration (when no microbatch size and
 * parallel split fits the global batch): it has no group, and every later call succeeds with
 * empty results.  Errors: MIST_E_INVALID (a descriptor), MIST_E_RANGE (a group of 2^32 - 1 or
 * more configurations: local ids are 32-bit), MIST_E_NOMEM, MIST_E_DEVICE. */
mist_status mist_space_create(const mist_model_desc* m, const mist_hw_desc* hw, int32_t n_hw,
                              const mist_space_desc* s, const mist_allocator* alloc,
                              mist_space** out);

/* Enqueues the evaluation of every configuration (cost model, feasibility filter, per
 * bucket and per group reductions; Sec. 5.3, Eq. 4-6, Algorithm 1) on hip_stream
 * (a hipStream_t; NULL = the null stream) and returns without waiting.  Re-runnable; each
 * run overwrites the previous results.  On a stream other than the one of the space's
 * previous evaluation or exact frontier, it first waits on the host for the work queued
 * there (the two share buffers).  Errors: MIST_E_INVALID, MIST_E_DEVICE. */
mist_status mist_eval_space(mist_space* S, void* hip_stream);

/* The intra-stage optimum of Eq. 4 (objective G*t + d, subject to the memory budget) per
 * candidate stage: waits for the last evaluation and writes, for groups g0..g0+n-1, the
 * feasible configuration of minimum obj (lowest id among equal obj) into host out[0..n-1]; a
 * group without a feasible configuration gets id MIST_NONE, obj +inf, bucket -1.
 * Errors: MIST_E_STATE (no evaluation yet), MIST_E_RANGE, MIST_E_DEVICE. */
mist_status mist_get_best(mist_space* S, int64_t g0, int64_t n, mist_result* out);

/* The time-vs-memory Pareto staircase that the inter-stage partitioner consumes (Eq. 3: each
 * stage's frontier over its memory use; here over 64 memory-budget buckets): waits for the
 * last evaluation and writes the staircase of group g into host out[0..*n_out-1] in
 * increasing bucket order: bucket j is on it when it holds a feasible configuration whose obj
 * is strictly below that of every lower bucket.  If cap
 * is too small returns MIST_E_RANGE with *n_out set to the required count. */
mist_status mist_get_pareto(mist_space* S, int64_t g, mist_result* out, int32_t cap,
                            int32_t* n_out);

/* Eq. 4 with sampled weights (Sec. 5.3, the intra-stage (t, d) frontier): waits for the last
 * evaluation and writes, for groups g0..g0+n-1 and each weight sample alpha_a of the space,
 * the feasible configuration minimising fma(alpha_a*G, t, (1-alpha_a)*d) (alpha_a*G and
 * 1-alpha_a each rounded once; lowest id among equal values) into host out[i*A + a], A =
 * n_alphas; obj holds that weighted value (+inf and id MIST_NONE when the group has no
 * feasible configuration).  Errors: MIST_E_STATE (no samples, or no evaluation yet),
 * MIST_E_RANGE, MIST_E_DEVICE. */
mist_status mist_get_alpha(mist_space* S, int64_t g0, int64_t n, mist_result* out);

/* Inter-stage planner (Sec. 5.3, Eq. 1-3), host only: among the candidate points pts[0..n-1]
 * of one hardware sample, chooses G, PP, the layer counts l_1..l_PP (summing to n_layers; stage
 * i draws from the points of group (G, PP, k = PP - i + 1, l_i)) and one point per stage so
 * that Eq. 2 is minimal (a dominance-pruned dynamic program over stages).  The plan chosen is
 * the exact minimum of Eq. 2 evaluated as (G-1)*max t_i + max_i (d_i + sum_{j>=i} t_j), the sums
 * taken from the last stage to the first (the form whose rounding the pruning respects; among
 * equal values, the smallest G, then PP).  out->F is that plan's value in stage order (the
 * field's form), which can differ from the stage-order minimum by the rounding of the two
 * sums, a few ulps.  pp = 0 allows every PP, otherwise only plans with PP = pp
 * (<= MIST_MAX_STAGES; points of larger PP are ignored).  Writes *out (found = 0 when no plan
 * exists).  Errors: MIST_E_INVALID. */
mist_status mist_plan_points(const mist_stage_point* pts, int64_t n, int32_t n_layers, int32_t pp,
                             mist_plan* out);

/* The planner on an evaluated space: every group of hardware sample hw contributes its best
 * configuration and, when the space has weight samples, the configuration each sample selects
 * (its points of the (t, d) frontier, Eq. 3-4); waits for the last evaluation, re-evaluates the
 * points' t and d on the device and calls mist_plan_points with the model's layer count.
 * Errors: MIST_E_STATE (no evaluation yet), MIST_E_RANGE (hw), MIST_E_DEVICE, MIST_E_NOMEM. */
mist_status mist_plan_pipeline(mist_space* S, int32_t hw, int32_t pp, mist_plan* out);

/* Exact time-vs-memory frontier of every group (the staircase without memory buckets): after
 * mist_eval_space, finds for each group the feasible configurations whose obj is strictly
 * below that of every configuration before them in (mem, obj, id) order.  A candidate pass
 * keeps only configurations that beat every lower bucket's minimum and are not dominated by
 * their bucket's winner (each tile writes them to a window of its own, the rest to a shared
 * overflow pool, and counts them; a tile whose candidates do not all find a place is evaluated
 * a second time, see cand_window); they are sorted by memory per group and scanned.  Waits for the evaluation and once more for the
 * candidate counts, then enqueues the rest on hip_stream.
 * Errors: MIST_E_STATE (no evaluation yet), MIST_E_RANGE (2^32 candidates or more),
 * MIST_E_NOMEM, MIST_E_DEVICE. */
mist_status mist_eval_pareto_exact(mist_space* S, void* hip_stream);

/* The exact frontier of group g in increasing memory (strictly decreasing obj) into host
 * out[0..*n_out-1]; returns MIST_E_RANGE with *n_out set when cap is too small.  Waits for
 * mist_eval_pareto_exact.  Errors: MIST_E_STATE, MIST_E_RANGE, MIST_E_DEVICE. */
mist_status mist_get_pareto_exact(mist_space* S, int64_t g, mist_result* out, int64_t cap, int64_t* n_out);

/* Sizes of the last exact frontier, for diagnostics and measurement: the candidates of the
 * candidate pass (all groups), those the pre-filter kept, the tiles the candidate pass
 * evaluated (those that may hold a candidate) and the tiles evaluated a second time because
 * a candidate found no place in its window or the overflow pool.  Waits for mist_eval_pareto_exact; any pointer may
 * be NULL.  Errors: MIST_E_INVALID, MIST_E_STATE, MIST_E_DEVICE, MIST_E_NOMEM. */
mist_status mist_exact_info(mist_space* S, int64_t* n_candidates, int64_t* n_kept, int32_t* n_tiles_live,
                            int32_t* n_tiles_again);

/* Per-group sizes of the last exact frontier, groups g0..g0+n-1: host candidates[i] (the
 * candidate pass's configurations of the group) and host kept[i] (those the pre-filter kept for
 * the sort and scan); either pointer may be NULL.  Waits for mist_eval_pareto_exact.
 * Errors: MIST_E_INVALID, MIST_E_STATE, MIST_E_RANGE, MIST_E_DEVICE, MIST_E_NOMEM. */
mist_status mist_exact_group_sizes(mist_space* S, int64_t g0, int64_t n, int64_t* candidates, int64_t* kept);

/* Raw per-bucket table of groups g0..g0+n-1: host ids[n*NB] and objs[n*NB] (MIST_NONE /
 * +inf for empty buckets) and host frontier masks[n] (bit j = bucket j on the staircase);
 * any output pointer may be NULL.  Waits for the last evaluation.  Errors as get_best. */
mist_status mist_get_buckets(mist_space* S, int64_t g0, int64_t n, uint64_t* ids, double* objs,
                             uint64_t* masks);

/* Sizes of the space: configurations, groups, buckets.  Any pointer may be NULL. */
mist_status mist_space_info(const mist_space* S, uint64_t* n_configs, int64_t* n_groups,
                            int32_t* n_buckets);

/* Key of group g (the (hw, G, PP, k, l) of one candidate stage, Sec. 5.3, and its id range)
 * into host *out.  The group-key query of the boundary; it carries a get_ prefix because the
 * name mist_group_key is the struct type's.  Errors: MIST_E_RANGE. */
mist_status mist_get_group_key(const mist_space* S, int64_t g, mist_group_key* out);

/* Decodes a global id into host *out (host-side arithmetic only).  Errors: MIST_E_RANGE. */
mist_status mist_decode(const mist_space* S, uint64_t id, mist_config* out);

/* Evaluates the configurations host ids[0..n-1] on the device with the same cost-model code
 * as mist_eval_space and writes host out[4*i..4*i+3] = t, d, mem, obj.  Synchronous on
 * hip_stream.  Errors: MIST_E_RANGE (an id >= the number of configurations), MIST_E_NOMEM,
 * MIST_E_DEVICE. */
mist_status mist_eval_ids(mist_space* S, const uint64_t* ids, int64_t n, double* out,
                          void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): mist_eval_ids without any allocation.  The ids and
 * results pass through a fixed 4 MiB device array of the library (one per GPU, held until the
 * process ends), so n is at most 104,857 per call; the space's device must be current.  It
 * calls no hipMalloc or hipFree (the host-to-device and device-to-host copies use the HIP
 * runtime's own staging for pageable host memory).  Calls that overlap on one GPU share the
 * array and race: issue them one at a time per GPU.  Synchronous on hip_stream.
 * Errors: MIST_E_INVALID (null argument, another device current), MIST_E_RANGE (more ids than
 * the array holds, or an id >= the number of configurations), MIST_E_DEVICE. */
mist_status mist_eval_ids_noalloc(mist_space* S, const uint64_t* ids, int64_t n, double* out, void* hip_stream);

/* Kernel timing.  mist_set_timing(S, 1) waits for pending work and starts recording HIP
 * events around the two kernels of every later mist_eval_space, on the evaluation stream;
 * mist_read_timing waits for the recorded evaluations and returns the summed durations (ms)
 * of the evaluation kernel and of the group-reduction kernel and their count, then starts a
 * new record.  mist_set_timing(S, 0) stops recording.  Errors: MIST_E_STATE (timing off),
 * MIST_E_DEVICE. */
mist_status mist_set_timing(mist_space* S, int32_t on);
mist_status mist_read_timing(mist_space* S, double* eval_ms, double* reduce_ms, int64_t* n_evals);

/* Tile t of the evaluation kernel: its group, the global id of its first configuration and its
 * configuration count (a tile covers consecutive ids of one group).  Errors: MIST_E_RANGE. */
mist_status mist_tile_info(const mist_space* S, int32_t t, int64_t* group, uint64_t* first_id, int64_t* n_configs);

/* Parity checks of the evaluation kernel itself (the cost model of Eq. 4-6 with Algorithm 1,
 * Sec. 5.2): runs the evaluation kernel's own per-configuration path (not the per-id path of
 * mist_eval_ids) over the listed tiles and writes, for every configuration of tiles[0..n-1] in
 * that order and in id order within a tile, six doubles into host out: t, d, mem, obj, the
 * bucket entry the kernel chose (0..NB-1 for a feasible configuration; NB..64 for an infeasible
 * one, which the reduction ignores) and the forms in which it evaluated Algorithm 1 for the
 * configuration, f1 + 8 * fs with f1 the first microbatch's form and fs the stable time's:
 * 1 compute and the larger host stream left after the second round (per-lane third row), 2 compute
 * finished in the second round (one third row for the wave), 3 the third row looked up per lane,
 * 4 the general rounds, 5 the all-zero configuration's closed form, 6 three rounds from an unknown
 * first pattern.  cap is the capacity of out in configurations.
 * Synchronous on hip_stream; allocates temporary device memory through the space's allocator.
 * Errors: MIST_E_INVALID, MIST_E_RANGE (a tile index, or cap too small), MIST_E_NOMEM,
 * MIST_E_DEVICE. */
mist_status mist_debug_eval_tiles(mist_space* S, const int32_t* tiles, int32_t n, double* out, int64_t cap,
                                  void* hip_stream);

/* Launch geometry of the evaluation kernel: tiles (work items, one wave each), threads per
 * tile, strips per full-size tile (a strip is the R^2 configurations sharing pair,
 * recomputed layers, ZeRO level, weight and gradient ratios). */
mist_status mist_launch_info(const mist_space* S, int64_t* n_tiles, int32_t* block,
                             int32_t* strips_per_tile);

/* ---------------------------------------------------------------------------------------
 * Calibration of the cost model's constants on the current device.  Mist estimates compute
 * time from an operator database benchmarked on the target hardware (Sec. 5.2.1) and fits one
 * slowdown factor per co-running combination and participant from benchmarked co-runs of
 * computation and communication kernels (Sec. 5.2.2, the fit after Algorithm 1).  The four
 * streams are those of Algorithm 1: 0 compute, 1 GPU-GPU, 2 host->device, 3 device->host.
 * --------------------------------------------------------------------------------------- */

#define MIST_CORUN_MAX_UNITS 256
#define MIST_CORUN_SAMPLES_PER_SHAPE 28 /* members of the 11 combinations of >= 2 streams */

/* One unit of work of each stream. */
typedef struct mist_corun_shape {
  int64_t gemm_m, gemm_n, gemm_k; /* compute: one rocBLAS bf16 GEMM D = A^T B (A k x m, B k x n,
                                     D m x n, column-major, fp32 accumulation), each in 1..2^31-1 */
  int64_t g2g_bytes;  /* GPU-GPU: one device-to-device copy by a kernel of g2g_blocks workgroups
                         (on one device this stands in for a collective's kernel: it occupies CUs
                         and HBM, not a link); a positive multiple of 16 */
  int64_t h2d_bytes;  /* host->device: one copy from pinned host memory, positive */
  int64_t d2h_bytes;  /* device->host: one copy into pinned host memory, positive */
} mist_corun_shape;

typedef struct mist_corun mist_corun;

/* Creates the benchmark's state on the current device: four streams of default priority plus
 * a control stream, device buffers and pinned host buffers large enough for every field of
 * *max, a rocBLAS handle and the events.  The operands hold pseudo-random values.  Errors:
 * MIST_E_INVALID, MIST_E_NOMEM, MIST_E_DEVICE. */
mist_status mist_corun_create(const mist_corun_shape* max, int32_t g2g_blocks, mist_corun** out);

/* Runs the streams of mask (bit j = stream j) together: every member waits for one common
 * start, then stream j runs units[j] (1..MIST_CORUN_MAX_UNITS; entries of non-members are
 * ignored) units of shape *sh back to back with an event before the first and after each, and
 * host t[j*stride + i] (i = 0..units[j]; stride > every units[j])
 * receives the events' times in seconds after the common start.  Synchronous.  Errors:
 * MIST_E_INVALID (mask, units, stride, or a shape field above the creation maximum),
 * MIST_E_DEVICE. */
mist_status mist_corun_run(mist_corun* C, int32_t mask, const mist_corun_shape* sh, const int32_t* units,
                           double* t, int32_t stride);

/* The all-running window of one run, host only: over the members j of mask the window is
 * [max_j t[j*stride], min_j t[j*stride + units[j]]]; host mean[j] receives the mean duration of
 * member j's units that lie entirely inside it and count[j] their number (NaN and 0 for
 * non-members and for members without such a unit).  Inside the window the running streams are
 * exactly those of mask, the situation a factor phi[mask][j] describes.  Errors:
 * MIST_E_INVALID (empty mask, units < 1, stride too small, decreasing times). */
mist_status mist_corun_reduce(int32_t mask, const double* t, int32_t stride, const int32_t* units,
                              double* mean, int32_t* count);

/* One benchmarked (combination, member, shape): mean unit times alone and inside the window. */
typedef struct mist_corun_sample {
  int32_t mask, stream, shape; /* shape: index into the shapes given to mist_corun_measure */
  int32_t units;               /* co-run units inside the window */
  double solo_s, corun_s;
} mist_corun_sample;

/* The co-run benchmark: for each shape k, every stream alone (units[j] = clamp(ceil(target_s /
 * first-run unit time), 3, MIST_CORUN_MAX_UNITS)), then each of the 11 combinations of two or
 * more streams with the same unit counts (once more with doubled counts if a member has no
 * unit inside the window).  A member that still has none was starved while the others ran: its
 * sample gets units = 0 and corun_s = the window's length, a lower bound of its unit time.
 * Writes MIST_CORUN_SAMPLES_PER_SHAPE samples per shape into host out, in shape, mask, stream
 * order.  Errors: MIST_E_RANGE (cap too small; *n_out receives the count), MIST_E_INVALID,
 * MIST_E_STATE (a window is empty: the streams never ran together), MIST_E_DEVICE. */
mist_status mist_corun_measure(mist_corun* C, const mist_corun_shape* shapes, int32_t n_shapes,
                               double target_s, mist_corun_sample* out, int32_t cap, int32_t* n_out);

/* Frees the benchmark's state.  NULL is accepted. */
mist_status mist_corun_destroy(mist_corun* C);

/* Fits the slowdown factors to benchmarked co-runs, host only: for every combination of two or
 * more streams and each member j, phi[mask*4 + j] = max(1, sum corun_s*solo_s / sum solo_s^2)
 * over its samples (the least-squares factor from solo to co-run unit time; a measured speed-up
 * is noise, the model's factors are slowdowns); every other entry of host phi[64] is 1.
 * Errors: MIST_E_INVALID (a sample whose stream is not in its mask or whose times are not
 * positive and finite, or a member of a combination without samples). */
mist_status mist_fit_phi(const mist_corun_sample* s, int64_t n, double* phi);

/* Algorithm 1 on one vector of stream times, host only: host x[4] (seconds, >= 0, finite) and
 * factors host phi[64] (phi[mask*4 + j], finite and >= 1 for the members of combinations of
 * two or more streams) give the overlapped time in *out, with the evaluation kernel's
 * arithmetic (psi = 1/phi rounded once; updates while two or more streams are non-zero).
 * Errors: MIST_E_INVALID. */
mist_status mist_interference(const double* phi, const double* x, double* out);

/* Operator database of one model on the current device: for each microbatch size mb[i] (n_mb
 * in 1..MIST_MAX_MB), times the forward GEMMs of one transformer layer at tensor parallelism tp
 * on mb[i]*seq tokens (query/key/value and output projections, the MLP's up (GPT) or gate+up
 * (Llama) and down projections; rocBLAS bf16, weights transposed), one warm-up and reps >= 1
 * timed runs, and writes host eta[i] = their FLOPs / median time / peak_flops and host sec[i] =
 * the median time.  The attention core is not timed; the cost model applies the same
 * efficiency to it.  Errors: MIST_E_INVALID (tp must divide heads, hidden and ffn), MIST_E_NOMEM,
 * MIST_E_DEVICE. */
mist_status mist_measure_eta(const mist_model_desc* m, const int32_t* mb, int32_t n_mb, int32_t tp,
                             double peak_flops, int32_t reps, double* eta, double* sec);

/* ---------------------------------------------------------------------------------------
 * Measurement support: an FP64 instruction-mix probe for reading the profiler's per-type FP64
 * instruction counters (which of them counts FP64 min, max and compare) against known counts.
 * --------------------------------------------------------------------------------------- */
#define MIST_PROBE_ADD 0
#define MIST_PROBE_MUL 1
#define MIST_PROBE_FMA 2
#define MIST_PROBE_MIN 3
#define MIST_PROBE_MAX 4
#define MIST_PROBE_CMP 5 /* v_cmp_lt_f64 */

/* Enqueues on hip_stream one kernel of n_threads threads (a positive multiple of 256) each of
 * which issues reps x 8 FP64 instructions of the given kind and no other FP64 arithmetic; it
 * reads device in[2 * n_threads] (operands; any finite values) and writes device
 * out[n_threads].  *n_instructions (may be NULL) receives the wave-level count of the probed
 * instruction: n_threads / 64 x reps x 8.  Errors: MIST_E_INVALID, MIST_E_DEVICE. */
mist_status mist_probe_fp64(int32_t kind, const double* in, uint64_t* out, int64_t n_threads, int32_t reps,
                            uint64_t* n_instructions, void* hip_stream);

/* Frees every buffer of the space (through its allocator).  NULL is accepted. */
mist_status mist_space_destroy(mist_space* S);

/* Message of the last failed call on this thread ("" if none). */
const char* mist_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MIST_H */
