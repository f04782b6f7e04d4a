// libmist host side: descriptor validation, space enumeration (groups, pairs, tiles),
// reciprocal / edge / interference tables, device buffers, and the C ABI of mist.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "mist.h"
#include "mist_internal.h"

using namespace mist;

namespace {

thread_local std::string g_error;

mist_status fail(mist_status code, const std::string& msg) {
  g_error = msg;
  return code;
}

mist_status fail_hip(hipError_t e, const char* what) {
  return fail(MIST_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Copies that accept an empty range (a space may have no group; a caller may ask for none).
hipError_t copy_sync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
  return bytes ? hipMemcpy(dst, src, bytes, kind) : hipSuccess;
}

hipError_t copy_async(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t st) {
  return bytes ? hipMemcpyAsync(dst, src, bytes, kind, st) : hipSuccess;
}

constexpr int64_t kExact = (int64_t)1 << 53;  // integers below this convert to double exactly
constexpr int64_t kStaticStrips = 512;        // strips per resident wave up to which a space is
                                              // cut into one tile per wave
constexpr int64_t kMinTileConfigs = 16384;    // configurations per tile of a larger space, at least
constexpr int64_t kMaxTiles = 131072;         // and tiles per space, at most
constexpr int64_t kWindowDiv = 8;             // exact frontier: candidate window of a tile,
                                              // 1/kWindowDiv of its configurations
constexpr int64_t kWindowSlots = (int64_t)1 << 27;  // and all windows together, at most
constexpr int64_t kPoolSlots = (int64_t)1 << 27;    // overflow pool of the candidate pass, at most
constexpr int64_t kTailPercent = 10;          // share of each group's strips in small tiles
constexpr int64_t kStripAlign = kWaveTile;    // strips per tile: a multiple of the wave

int popcount4(int v) { return (v & 1) + ((v >> 1) & 1) + ((v >> 2) & 1) + ((v >> 3) & 1); }

}  // namespace

struct mist_space {
  // copied descriptors
  mist_model_desc model;
  std::vector<mist_hw_desc> hw;
  int64_t D = 0, B = 0;
  std::vector<int32_t> mb;
  std::vector<double> ratio_om;  // r[0..R), om[0..R)
  int32_t R = 0, NB = 0, l_rule = 0;
  // enumeration
  std::vector<DevGroup> groups;
  std::vector<DevPair> pairs;
  std::vector<DevTile> tiles;
  std::vector<int32_t> tile_order;  // work item -> tile (build_tile_order)
  std::vector<DevHw> hws;
  std::vector<int32_t> pk_group;  // group of each pair-constant entry
  DevModel dm;
  uint64_t n_configs = 0;
  int32_t strips_per_tile = 0;
  // memory
  mist_allocator alloc{};
  bool custom_alloc = false;
  std::vector<void*> dev_buffers;
  DevGroup* d_groups = nullptr;
  DevPair* d_pairs = nullptr;
  DevTile* d_tiles = nullptr;
  int32_t* d_tile_order = nullptr;
  DevHw* d_hws = nullptr;
  double* d_ratio = nullptr;
  PairK* d_pk = nullptr;
  int32_t* d_pk_group = nullptr;
  int32_t* d_work = nullptr;
  int32_t eval_grid = 0;
  int64_t tile_configs = 0;  // configurations per full-size tile, at least
  int32_t max_blocks = 0;    // cap on the evaluation grid (0: none)
  int32_t cand_window = 0;   // exact frontier: window divisor (0: automatic)
  int32_t max_group_tiles = 0;  // tiles (full-size and small) of the largest group
  double* d_part_obj = nullptr;
  uint64_t* d_part_id = nullptr;
  double* d_bucket_obj = nullptr;
  uint64_t* d_bucket_id = nullptr;
  double* d_best_obj = nullptr;
  uint64_t* d_best_id = nullptr;
  uint64_t* d_frontier = nullptr;
  // weight samples of Eq. 4 (A = 0: off)
  int32_t A = 0;
  std::vector<double> alphas, betas;  // alpha_a and 1 - alpha_a
  double* d_alpha = nullptr;
  double* d_beta = nullptr;
  double* d_part_aobj = nullptr;
  uint64_t* d_part_aid = nullptr;
  double* d_alpha_obj = nullptr;
  uint64_t* d_alpha_id = nullptr;
  int32_t cus = 0;
  int32_t device = 0;  // the HIP device the space was created on
  // exact frontier (mist_eval_pareto_exact)
  bool exact_done = false;
  bool exact_launched = false;  // some call enqueued uploads of the host offset tables
  hipStream_t exact_stream = nullptr;
  FiltEntry* d_filt = nullptr;
  int32_t* d_cnt_tile = nullptr;
  int64_t* d_tile_off = nullptr;
  int64_t* d_tile_end = nullptr;
  int32_t* d_list = nullptr;
  uint8_t* d_live = nullptr;  // per tile: may hold a candidate
  // Overflow pool of the candidate pass: candidates past their tile's window.
  unsigned long long* d_pool_count = nullptr;
  int64_t pool_cap = 0;
  uint64_t *d_pool_key = nullptr, *d_pool_id = nullptr;
  double* d_pool_obj = nullptr;
  int32_t *d_pool_tile = nullptr, *d_pool_rank = nullptr;
  uint8_t* d_tile_drop = nullptr;  // per tile: a candidate found no place (evaluated again)
  uint8_t* h_drop = nullptr;
  unsigned long long* h_pool_count = nullptr;
  int64_t n_pooled = 0;  // candidates the last call placed through the pool
  // Candidate windows: tile t writes to slots [slab_begin[t], slab_begin[t+1]) first.
  std::vector<int64_t> h_slab_begin;
  int64_t* d_slab_begin = nullptr;
  uint64_t *d_slab_key = nullptr, *d_slab_id = nullptr;
  double* d_slab_obj = nullptr;
  int64_t* d_seg = nullptr;
  int64_t* d_seg_end = nullptr;  // end of each group's candidates after the pre-filter
  int64_t* d_front_cnt = nullptr;
  // Pinned host staging of the per-tile counts and the offset tables (copies to and from it
  // run without a staging step); allocated by the first exact frontier, freed by destroy.
  void* h_pinned = nullptr;
  int32_t* h_cnt = nullptr;
  int64_t* h_tile_off = nullptr;
  int64_t* h_tile_end = nullptr;
  int64_t* h_seg = nullptr;
  int32_t* h_list = nullptr;
  int32_t n_list = 0;
  int64_t cand_cap = 0, n_cand = 0;
  int32_t n_rerun = 0;  // tiles the last call evaluated a second time
  uint64_t *d_cand_key = nullptr, *d_cand_id = nullptr, *d_key_sorted = nullptr;
  double* d_cand_obj = nullptr;
  uint32_t *d_idx_in = nullptr, *d_idx_out = nullptr;
  uint64_t *d_front_key = nullptr, *d_front_id = nullptr;
  double* d_front_obj = nullptr;
  // state
  bool evaluated = false;
  hipStream_t stream = nullptr;
  bool timing = false;
  std::vector<hipEvent_t> events;  // pool; three per timed evaluation
  size_t events_used = 0;
};

namespace {

// A device buffer owned by the space; `st` is the stream of its first use (see mist_allocator).
void* dev_alloc(mist_space* S, size_t bytes, hipStream_t st) {
  if (bytes == 0) bytes = 256;
  void* p = nullptr;
  if (S->custom_alloc) {
    p = S->alloc.alloc(bytes, (void*)st, S->alloc.ctx);
  } else if (hipMalloc(&p, bytes) != hipSuccess) {
    p = nullptr;
  }
  if (p) S->dev_buffers.push_back(p);
  return p;
}

void dev_free_one(mist_space* S, void* p) {
  if (!p) return;
  for (size_t i = 0; i < S->dev_buffers.size(); ++i)
    if (S->dev_buffers[i] == p) {
      S->dev_buffers.erase(S->dev_buffers.begin() + (long)i);
      break;
    }
  if (S->custom_alloc) S->alloc.free(p, S->alloc.ctx);
  else (void)hipFree(p);
}

void dev_free_all(mist_space* S) {
  for (void* p : S->dev_buffers) {
    if (S->custom_alloc) S->alloc.free(p, S->alloc.ctx);
    else (void)hipFree(p);
  }
  S->dev_buffers.clear();
}

// A temporary device buffer released at scope exit.
struct TempBuf {
  mist_space* S;
  void* p = nullptr;
  TempBuf(mist_space* s, size_t bytes, hipStream_t st) : S(s) {
    if (bytes == 0) bytes = 256;
    if (S->custom_alloc) p = S->alloc.alloc(bytes, (void*)st, S->alloc.ctx);
    else if (hipMalloc(&p, bytes) != hipSuccess) p = nullptr;
  }
  ~TempBuf() {
    if (!p) return;
    if (S->custom_alloc) S->alloc.free(p, S->alloc.ctx);
    else (void)hipFree(p);
  }
};

bool tp_admissible(const mist_model_desc& m, int64_t per_stage, int64_t tp) {
  if (per_stage % tp || m.heads % tp || m.ffn % tp) return false;
  if (tp <= m.kv_heads) return m.kv_heads % tp == 0;
  return tp % m.kv_heads == 0;
}

std::string validate(const mist_model_desc* m, const mist_hw_desc* hw, int32_t n_hw,
                     const mist_space_desc* s) {
  if (!m || !hw || !s) return "null descriptor";
  if (n_hw < 1) return "n_hw must be >= 1";
  if (m->arch != MIST_ARCH_GPT && m->arch != MIST_ARCH_LLAMA) return "unknown arch";
  if (m->n_layers < 1 || m->hidden < 1 || m->heads < 1 || m->kv_heads < 1 || m->ffn < 1 ||
      m->seq < 1 || m->vocab < 1 || m->bytes_w < 1 || m->bytes_opt < 1)
    return "model sizes must be positive";
  if (m->flash != 0 && m->flash != 1) return "flash must be 0 or 1";
  if (m->hidden % m->heads) return "hidden must be a multiple of heads";
  if (m->heads % m->kv_heads) return "heads must be a multiple of kv_heads";
  // Magnitude bounds (far beyond any physical value) under which every non-zero stream time is
  // at least 2^-363 and at most 2^500: a difference of two distinct scaled times then exceeds
  // 2^-415, and dividing it by a factor of at most 2^100 cannot round to zero, which the
  // evaluation kernel's second interference round relies on (a stream keeps running exactly when
  // its scaled time exceeds the overlap).
  const double lo_rate = 0x1p-200, hi_rate = 0x1p200, lo_eff = 0x1p-100, hi_eff = 0x1p100;
  for (int32_t i = 0; i < n_hw; ++i) {
    const mist_hw_desc& h = hw[i];
    const double v[4] = {h.flops, h.mem_bytes, h.pcie_bw, h.link_bw};
    for (double x : v)
      if (!(x > 0.0) || !std::isfinite(x)) return "hardware rates and memory must be positive and finite";
    if (!(h.flops >= lo_rate && h.flops <= hi_rate && h.pcie_bw >= lo_rate && h.pcie_bw <= hi_rate &&
          h.link_bw >= lo_rate && h.link_bw <= hi_rate))
      return "flops, pcie_bw and link_bw must lie in [2^-200, 2^200]";
    if (!(h.eta_max >= 0.0) || !std::isfinite(h.eta_max) || !(h.n_half >= 0.0) || !std::isfinite(h.n_half))
      return "eta_max and n_half must be non-negative and finite";
    if (h.eta_max != 0.0 && !(h.eta_max >= lo_eff && h.eta_max <= hi_eff)) return "eta_max must be 0 or in [2^-100, 2^100]";
    if (!(h.n_half <= hi_eff)) return "n_half must be at most 2^100";
    if (h.eta_max == 0.0 && s && s->mb && s->n_mb >= 1 && s->n_mb <= MIST_MAX_MB)
      for (int32_t j = 0; j < s->n_mb; ++j)
        if (!(h.eta_tab[j] >= lo_eff && h.eta_tab[j] <= hi_eff))
          return "with eta_max = 0 every eta_tab entry of the microbatch list must lie in [2^-100, 2^100]";
    for (int mask = 0; mask < 16; ++mask) {
      if (popcount4(mask) < 2) continue;
      for (int j = 0; j < 4; ++j)
        if ((mask >> j & 1) && !(h.phi[mask][j] >= 1.0 && std::isfinite(h.phi[mask][j])))
          return "slowdown factors must be finite and >= 1";
        else if ((mask >> j & 1) && !(h.phi[mask][j] <= hi_eff))
          return "slowdown factors must be at most 2^100";
    }
  }
  if (s->n_devices < 1 || s->global_batch < 1) return "n_devices and global_batch must be positive";
  if (s->n_mb < 1 || s->n_mb > MIST_MAX_MB || !s->mb) return "n_mb out of range";
  for (int32_t i = 0; i < s->n_mb; ++i)
    if (s->mb[i] < 1 || (i && s->mb[i] <= s->mb[i - 1])) return "mb must be ascending and >= 1";
  if (s->n_ratios < 1 || s->n_ratios > MIST_MAX_RATIOS || !s->ratios) return "n_ratios out of range";
  for (int32_t i = 0; i < s->n_ratios; ++i)
    if (!(s->ratios[i] >= 0.0 && s->ratios[i] <= 1.0) || (i && !(s->ratios[i] > s->ratios[i - 1])))
      return "ratios must be strictly ascending in [0, 1]";
    else if (s->ratios[i] != 0.0 && !(s->ratios[i] >= 0x1p-100))
      return "a non-zero ratio must be at least 2^-100";
  if (s->n_buckets < 1 || s->n_buckets > MIST_MAX_BUCKETS) return "n_buckets out of range";
  if (s->l_rule != MIST_L_FULL && s->l_rule != MIST_L_BALANCED) return "unknown l_rule";
  if (s->n_alphas < 0 || s->n_alphas > MIST_MAX_ALPHAS || (s->n_alphas > 0 && !s->alphas))
    return "n_alphas out of range";
  if (s->tile_configs < 0 || s->tile_configs > ((int64_t)1 << 40) || s->max_blocks < 0 || s->cand_window < 0)
    return "tile_configs, max_blocks and cand_window must be non-negative";
  for (int32_t i = 0; i < s->n_alphas; ++i)
    if (!(s->alphas[i] >= 0.0 && s->alphas[i] <= 1.0)) return "weight samples must lie in [0, 1]";
  return "";
}

// Largest integer quantities of the cost model for a (stage, pair); they must convert to
// double exactly.
bool counts_exact(const mist_model_desc& m, int64_t PP, int64_t l, int64_t b, int64_t tp,
                  int64_t dp, int64_t G) {
  // Work in long double-free int64 with overflow guards through __int128.
  const __int128 h = m.hidden, s = m.seq, V = m.vocab, f = m.ffn, bw = m.bytes_w, bo = m.bytes_opt;
  const __int128 dh = h / m.heads;
  const __int128 hkvr = tp <= m.kv_heads ? (__int128)m.kv_heads * dh / tp : dh;
  const __int128 Pq = 2 * h * h, Pm = (m.arch == MIST_ARCH_GPT ? 2 : 3) * h * f;
  const __int128 Psi = (Pq + Pm) / tp + 2 * h * hkvr + (m.arch == MIST_ARCH_GPT ? 4 * h : 2 * h);
  const __int128 Vr = (V + tp - 1) / tp;
  const __int128 Pe = Vr * h + s * h, Ph = Vr * h + 2 * h;
  const __int128 Pst = l * Psi + Pe + Ph;
  const __int128 Pbuf = Psi > Pe ? (Psi > Ph ? Psi : Ph) : (Pe > Ph ? Pe : Ph);
  const __int128 atok = 4 * h + (2 * h + 3 * f) / tp + 2 * hkvr + (__int128)m.heads * s / tp;
  const __int128 afull = (__int128)b * s * bw * atok;
  const __int128 ftok = 2 * ((Pq + Pm) / tp + 2 * h * hkvr) + 4 * s * h / tp;
  const __int128 ke = PP < G ? PP : G;
  const __int128 vals[] = {Pst * bo, Pst * bw * dp, 2 * Pbuf * bo, 2 * afull, ke * (l * afull),
                           (__int128)b * s * ftok, 3 * 2 * (__int128)b * s * h * Vr,
                           4 * (__int128)b * s * Vr, 2 * (__int128)b * s * h * bw * tp,
                           (__int128)(4 * l + 2 * l), (__int128)(3 * l + l)};
  for (__int128 v : vals)
    if (v >= kExact || v < 0) return false;
  return true;
}

// Enumerates the space.  On failure returns the message and sets *code: MIST_E_RANGE for a
// space beyond the sizes the kernels index (a group's local ids are 32-bit, and 0xFFFFFFFF
// marks an empty bucket), MIST_E_INVALID otherwise.
std::string enumerate(mist_space* S, mist_status* code) {
  *code = MIST_E_INVALID;
  const mist_model_desc& m = S->model;
  const int64_t L = m.n_layers;
  const int64_t R = S->R;
  const uint64_t per_unit = 4ull * (uint64_t)(R * R * R * R);
  uint64_t base = 0;
  S->groups.clear();
  S->pairs.clear();
  for (int32_t ih = 0; ih < (int32_t)S->hw.size(); ++ih) {
    for (int64_t PP = 1; PP <= S->D; ++PP) {
      if (S->D % PP || PP > L) continue;
      const int64_t per_stage = S->D / PP;
      struct Cand { int64_t G; DevPair p; };
      std::vector<Cand> cand;
      for (int32_t bi = 0; bi < (int32_t)S->mb.size(); ++bi) {
        const int64_t b = S->mb[bi];
        for (int64_t tp = 1; tp <= per_stage; ++tp) {
          if (!tp_admissible(m, per_stage, tp)) continue;
          const int64_t dp = per_stage / tp;
          if (S->B % (b * dp)) continue;
          DevPair p;
          p.b = (int32_t)b;
          p.tp = (int32_t)tp;
          p.dp = (int32_t)dp;
          p.mb = bi;
          p.inv_dp = 1.0 / (double)dp;
          cand.push_back({S->B / (b * dp), p});
        }
      }
      std::vector<int64_t> Gs;
      for (const Cand& c : cand) {
        bool seen = false;
        for (int64_t g : Gs) seen = seen || g == c.G;
        if (!seen) Gs.push_back(c.G);
      }
      std::sort(Gs.begin(), Gs.end());
      std::vector<int64_t> ls;
      if (S->l_rule == MIST_L_FULL) {
        if (PP == 1) ls.push_back(L);
        else for (int64_t l = 1; l <= L - PP + 1; ++l) ls.push_back(l);
      } else {
        ls.push_back(L / PP);
        if ((L + PP - 1) / PP != L / PP) ls.push_back((L + PP - 1) / PP);
      }
      for (int64_t G : Gs) {
        std::vector<DevPair> ps;
        for (const Cand& c : cand)
          if (c.G == G) ps.push_back(c.p);
        std::sort(ps.begin(), ps.end(), [](const DevPair& x, const DevPair& y) {
          return x.b < y.b || (x.b == y.b && x.tp < y.tp);
        });
        if (G > INT32_MAX) return "G too large";
        for (const DevPair& p : ps)
          for (int64_t l : ls)
            if (!counts_exact(m, PP, l, p.b, p.tp, p.dp, G))
              return "model too large: a cost-model count exceeds 2^53";
        const int32_t pair_begin = (int32_t)S->pairs.size();
        S->pairs.insert(S->pairs.end(), ps.begin(), ps.end());
        for (int64_t k = 1; k <= PP; ++k) {
          for (int64_t l : ls) {
            DevGroup g{};
            g.base = base;
            g.hw = ih;
            g.G = (int32_t)G;
            g.PP = (int32_t)PP;
            g.k = (int32_t)k;
            g.l = (int32_t)l;
            g.pair_begin = pair_begin;
            g.n_pairs = (int32_t)ps.size();
            const uint64_t units = (uint64_t)ps.size() * (uint64_t)(l + 1);
            // Local ids are 32-bit and 0xFFFFFFFF marks an empty bucket: a group holds fewer
            // than 2^32 - 1 configurations.
            const bool big = units > ((uint64_t)UINT32_MAX - 1) / per_unit;
            const uint64_t size = big ? 0 : units * per_unit;
            if (big || size >= (uint64_t)UINT32_MAX) {
              *code = MIST_E_RANGE;
              char msg[200];
              std::snprintf(msg, sizeof msg,
                            "group too large: %llu (pair, recomputed layers) units x %llu configurations "
                            "(PP %lld, G %lld, l %lld); a group holds at most 2^32 - 2 configurations",
                            (unsigned long long)units, (unsigned long long)per_unit, (long long)PP,
                            (long long)G, (long long)l);
              return msg;
            }
            if (base > UINT64_MAX - size) {
              *code = MIST_E_RANGE;
              return "space too large: 2^64 or more configurations";
            }
            base += size;
            S->groups.push_back(g);
          }
        }
      }
    }
  }
  S->n_configs = base;
  if (S->groups.size() > (size_t)INT32_MAX) return "too many groups";

  // Pair-constant entries, group-major.
  S->pk_group.clear();
  for (size_t gi = 0; gi < S->groups.size(); ++gi) {
    S->groups[gi].pk_begin = (int32_t)S->pk_group.size();
    for (int32_t p = 0; p < S->groups[gi].n_pairs; ++p) S->pk_group.push_back((int32_t)gi);
    if (S->pk_group.size() > (size_t)INT32_MAX) return "too many pairs";
  }

  // Strips per group (a strip is one (pair, c, z, wo, go) combination with its R x R
  // configurations); tiles are cut once the device's resident wave count is known.
  const uint64_t per_unit_strips = 4ull * (uint64_t)(R * R);
  for (const DevGroup& g : S->groups) {
    const uint64_t st = (uint64_t)g.n_pairs * (uint64_t)(g.l + 1) * per_unit_strips;
    if (st > (uint64_t)INT32_MAX) {  // strip indices are int32 (reached only with one ratio)
      *code = MIST_E_RANGE;
      return "group too large: 2^31 or more strips";
    }
  }

  // Per-hardware tables (host divisions, each correctly rounded).
  S->hws.assign(S->hw.size(), DevHw{});
  for (size_t i = 0; i < S->hw.size(); ++i) {
    const mist_hw_desc& h = S->hw[i];
    DevHw& d = S->hws[i];
    d.iF = 1.0 / h.flops;
    d.iP = 1.0 / h.pcie_bw;
    d.iL = 1.0 / h.link_bw;
    d.M = h.mem_bytes;
    // floor(mem * kNB) is min{j : mem <= E_j} or one below it (the margin 2^-40 exceeds
    // every rounding error involved and is far below a bucket width), so one comparison
    // with E_j settles the bucket.
    d.kNB = ((double)S->NB / h.mem_bytes) * (1.0 - 0x1p-40);
    for (int j = 0; j < MIST_MAX_MB; ++j) d.ieta[j] = 0.0;
    for (size_t j = 0; j < S->mb.size(); ++j) {
      if (h.eta_max == 0.0) {  // measured efficiency of this microbatch size
        d.ieta[j] = 1.0 / h.eta_tab[j];
        continue;
      }
      const double bs = (double)((int64_t)S->mb[j] * m.seq);
      d.ieta[j] = (bs + h.n_half) / (h.eta_max * bs);
    }
    const double inf = std::numeric_limits<double>::infinity();
    for (int j = 0; j < MIST_MAX_BUCKETS; ++j)
      d.edge[j] = j < S->NB ? (h.mem_bytes * (double)(j + 1)) / (double)S->NB : inf;
    d.edge[S->NB - 1] = h.mem_bytes;
    for (int mask = 0; mask < 16; ++mask)
      for (int j = 0; j < 4; ++j) {
        const bool update = popcount4(mask) >= 2;
        const bool member = (mask >> j) & 1;
        d.itab[mask][j] = !update ? 1.0 : (member ? h.phi[mask][j] : inf);
        d.itab[mask][4 + j] = (update && member) ? 1.0 / h.phi[mask][j] : 1.0;
      }
  }
  const int64_t hd = m.hidden;
  S->dm.h = hd;
  S->dm.heads = m.heads;
  S->dm.kv = m.kv_heads;
  S->dm.f = m.ffn;
  S->dm.s = m.seq;
  S->dm.V = m.vocab;
  S->dm.bw = m.bytes_w;
  S->dm.bo = m.bytes_opt;
  S->dm.gpt = m.arch == MIST_ARCH_GPT ? 1 : 0;
  S->dm.flash = m.flash;
  return "";
}

template <class T>
mist_status upload(mist_space* S, T** dst, const std::vector<T>& src, const char* what) {
  *dst = (T*)dev_alloc(S, src.size() * sizeof(T), nullptr);
  if (!*dst) return fail(MIST_E_NOMEM, std::string("device allocation failed: ") + what);
  if (src.empty()) return MIST_OK;
  const hipError_t e = copy_sync(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail_hip(e, what);
  return MIST_OK;
}

mist::EvalArgs eval_args(const mist_space* S) {
  EvalArgs a{};
  a.m = S->dm;
  a.groups = S->d_groups;
  a.pairs = S->d_pairs;
  a.tiles = S->d_tiles;
  a.tile_order = S->d_tile_order;
  a.hws = S->d_hws;
  a.ratio = S->d_ratio;
  a.R = S->R;
  a.NB = S->NB;
  a.n_tiles = (int32_t)S->tiles.size();
  a.n_groups = (int64_t)S->groups.size();
  a.n_configs = S->n_configs;
  a.part_obj = S->d_part_obj;
  a.part_id = S->d_part_id;
  a.pk = S->d_pk;
  a.pk_group = S->d_pk_group;
  a.n_pk = (int32_t)S->pk_group.size();
  a.work = S->d_work;
  a.n_alpha = S->A;
  a.alpha = S->d_alpha;
  a.beta = S->d_beta;
  a.part_aobj = S->d_part_aobj;
  a.part_aid = S->d_part_aid;
  return a;
}

mist_status wait_results(mist_space* S) {
  if (!S->evaluated) return fail(MIST_E_STATE, "mist_eval_space has not been called");
  const hipError_t e = hipStreamSynchronize(S->stream);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  return MIST_OK;
}

void decode_host(const mist_space* S, uint64_t id, mist_config* c) {
  size_t lo = 0, hi = S->groups.size();
  while (hi - lo > 1) {
    const size_t mid = (lo + hi) / 2;
    if (S->groups[mid].base <= id) lo = mid;
    else hi = mid;
  }
  const DevGroup& g = S->groups[lo];
  const uint64_t R = (uint64_t)S->R;
  uint64_t v = id - g.base;
  c->ao_idx = (int32_t)(v % R); v /= R;
  c->oo_idx = (int32_t)(v % R); v /= R;
  c->go_idx = (int32_t)(v % R); v /= R;
  c->wo_idx = (int32_t)(v % R); v /= R;
  c->zero = (int32_t)(v % 4); v /= 4;
  c->ckpt = (int32_t)(v % (uint64_t)(g.l + 1));
  const int32_t p = (int32_t)(v / (uint64_t)(g.l + 1));
  const DevPair& pr = S->pairs[g.pair_begin + p];
  c->hw = g.hw; c->G = g.G; c->PP = g.PP; c->k = g.k; c->l = g.l;
  c->b = pr.b; c->tp = pr.tp; c->dp = pr.dp;
  c->wo = S->ratio_om[c->wo_idx];
  c->go = S->ratio_om[c->go_idx];
  c->oo = S->ratio_om[c->oo_idx];
  c->ao = S->ratio_om[c->ao_idx];
}

// Device evaluation of ids for result extraction: out[4*i..] = t, d, mem, obj.
mist_status eval_ids_impl(mist_space* S, const uint64_t* ids, int64_t n, double* out, hipStream_t st) {
  if (n == 0) return MIST_OK;
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] >= S->n_configs) return fail(MIST_E_RANGE, "id out of range");
  TempBuf dids(S, (size_t)n * sizeof(uint64_t), st);
  TempBuf dout(S, (size_t)n * 4 * sizeof(double), st);
  if (!dids.p || !dout.p) return fail(MIST_E_NOMEM, "device allocation failed: eval_ids");
  // The temporary buffers go back to the allocator when this returns: on every path the
  // stream is drained first.
  auto drained = [&](mist_status code) {
    (void)hipStreamSynchronize(st);
    return code;
  };
  hipError_t e = copy_async(dids.p, ids, (size_t)n * sizeof(uint64_t), hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return drained(fail_hip(e, "hipMemcpyAsync ids"));
  const int rc = launch_eval_ids(eval_args(S), (const uint64_t*)dids.p, n, (double*)dout.p, st);
  if (rc) return drained(fail_hip((hipError_t)rc, "eval_ids launch"));
  e = copy_async(out, dout.p, (size_t)n * 4 * sizeof(double), hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return drained(fail_hip(e, "hipMemcpyAsync out"));
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  return MIST_OK;
}

int32_t bucket_host(const mist_space* S, const DevHw& h, double mem) {
  for (int32_t j = 0; j < S->NB; ++j)
    if (mem <= h.edge[j]) return j;
  return -1;
}

mist_status fill_results(mist_space* S, const uint64_t* ids, const double* objs, int64_t n, mist_result* out) {
  std::vector<uint64_t> want;
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] != MIST_NONE) want.push_back(ids[i]);
  std::vector<double> vals(want.size() * 4);
  mist_status rc = eval_ids_impl(S, want.data(), (int64_t)want.size(), vals.data(), S->stream);
  if (rc) return rc;
  size_t w = 0;
  for (int64_t i = 0; i < n; ++i) {
    mist_result& r = out[i];
    std::memset(&r, 0, sizeof(r));
    r.id = ids[i];
    r.obj = objs[i];
    if (ids[i] == MIST_NONE) {
      r.t = r.d = r.mem = std::numeric_limits<double>::infinity();
      r.bucket = -1;
      r.cfg.hw = -1;
      continue;
    }
    r.t = vals[4 * w + 0];
    r.d = vals[4 * w + 1];
    r.mem = vals[4 * w + 2];
    if (vals[4 * w + 3] != objs[i]) return fail(MIST_E_DEVICE, "re-evaluated objective differs");
    ++w;
    decode_host(S, r.id, &r.cfg);
    r.bucket = bucket_host(S, S->hws[r.cfg.hw], r.mem);
  }
  return MIST_OK;
}

}  // namespace

namespace {

// Tiles: contiguous strips of one group, at most strips_per_tile each (a multiple of the wave
// width).  Every wave of the persistent evaluation grid takes tile number (its global wave
// index) first and claims further tiles from the device counter, in tile order.  A space of
// at most kStaticStrips strips per resident wave is cut into about one tile per resident wave,
// so that no claim is made.  A larger one is cut into tiles of at least the space's
// tile_configs configurations (kMinTileConfigs unless the descriptor asks for another size;
// claims on one counter serialize) and at most kMaxTiles tiles; the last
// kTailPercent percent of a group's strips (rounded up to its last full-size tile) go into
// tiles a quarter of that size, placed after all full-size tiles, so that the waves that
// finish last wait for a small tile.
std::string build_tiles(mist_space* S, int64_t resident_waves) {
  const uint64_t per_unit_strips = 4ull * (uint64_t)(S->R * S->R);
  uint64_t total_strips = 0;
  for (const DevGroup& g : S->groups) total_strips += (uint64_t)g.n_pairs * (uint64_t)(g.l + 1) * per_unit_strips;
  const uint64_t W = (uint64_t)std::max<int64_t>(1, resident_waves);
  const uint64_t R2 = (uint64_t)(S->R * S->R);
  const auto align = [](uint64_t v) {
    v = (v + kStripAlign - 1) / kStripAlign * kStripAlign;
    if (v < (uint64_t)kStripAlign) v = kStripAlign;
    if (v > (uint64_t)INT32_MAX / 2) v = (uint64_t)INT32_MAX / 2 / kStripAlign * kStripAlign;
    return v;
  };
  const bool single = total_strips <= W * (uint64_t)kStaticStrips;
  uint64_t spt;
  if (single)
    spt = align((total_strips + W - 1) / W);
  else
    spt = align(std::max<uint64_t>(((uint64_t)S->tile_configs + R2 - 1) / R2,
                                   (total_strips + (uint64_t)kMaxTiles - 1) / (uint64_t)kMaxTiles));
  const uint64_t spt_tail = single ? spt : align(spt / 4);
  S->strips_per_tile = (int32_t)spt;
  S->tiles.clear();
  std::vector<DevTile> tail;
  for (size_t gi = 0; gi < S->groups.size(); ++gi) {
    DevGroup& g = S->groups[gi];
    const int64_t strips = (int64_t)g.n_pairs * (g.l + 1) * (int64_t)per_unit_strips;
    const int64_t split = single ? strips : strips * (100 - kTailPercent) / 100 / (int64_t)spt * (int64_t)spt;
    g.tile_begin = (int32_t)S->tiles.size();
    for (int64_t u = 0; u < split; u += (int64_t)spt) {
      DevTile t{};
      t.group = (int32_t)gi;
      t.strip_begin = (int32_t)u;
      t.strip_end = (int32_t)std::min<int64_t>(split, u + (int64_t)spt);
      S->tiles.push_back(t);
    }
    g.n_tiles = (int32_t)S->tiles.size() - g.tile_begin;
    g.tail_begin = (int32_t)tail.size();  // offset into the small tiles until they are appended
    for (int64_t u = split; u < strips; u += (int64_t)spt_tail) {
      DevTile t{};
      t.group = (int32_t)gi;
      t.strip_begin = (int32_t)u;
      t.strip_end = (int32_t)std::min<int64_t>(strips, u + (int64_t)spt_tail);
      tail.push_back(t);
    }
    g.n_tail = (int32_t)tail.size() - g.tail_begin;
    if (S->tiles.size() + tail.size() > (size_t)INT32_MAX / 2) return "too many tiles";  // + waves fits int
  }
  const int32_t full = (int32_t)S->tiles.size();
  for (DevGroup& g : S->groups) g.tail_begin += full;
  S->tiles.insert(S->tiles.end(), tail.begin(), tail.end());
  return "";
}

// Work items of the persistent evaluation grid in tile order per XCD.  Item i < n_waves is the
// first tile of wave i, whose block b = i / kWaves runs on XCD b mod kClaimCounters (blocks are
// dealt to the XCDs in turn); item n_waves + x + kClaimCounters * c is claim c on counter x, which
// the waves of XCD x draw from first.  Each XCD's items are given a contiguous range of the
// full-size tiles followed by a contiguous range of the small ones, in proportion to its item
// count: the pair constants, group records and hardware tables of neighbouring tiles are then
// reused from that XCD's L2, and each XCD still ends on small tiles.  Any permutation gives the
// same results; this one only decides which tiles share a cache.  Spaces of at most one tile
// per wave need no claims and keep item x = tile x.
std::string build_tile_order(mist_space* S, int64_t n_waves, int32_t n_full) {
  const int64_t n = (int64_t)S->tiles.size();
  S->tile_order.resize((size_t)n);
  for (int64_t i = 0; i < n; ++i) S->tile_order[(size_t)i] = (int32_t)i;
  if (n <= n_waves) return "";
  int64_t cnt[kClaimCounters] = {};
  for (int64_t i = 0; i < n_waves; ++i) ++cnt[(i / kWaves) % kClaimCounters];
  for (int64_t i = n_waves; i < n; ++i) ++cnt[(i - n_waves) % kClaimCounters];
  // XCD x takes full-size tiles [fc[x], fc[x+1]) and small tiles n_full + [sc[x], sc[x+1]); both
  // cumulative counts are non-decreasing and fc[x+1] - fc[x] + sc[x+1] - sc[x] = cnt[x].
  int64_t fc[kClaimCounters + 1], sc[kClaimCounters + 1], cum = 0;
  for (int x = 0; x <= kClaimCounters; ++x) {
    fc[x] = (int64_t)((__int128)n_full * cum / n);
    sc[x] = cum - fc[x];
    if (x < kClaimCounters) cum += cnt[x];
  }
  int64_t pos[kClaimCounters] = {};
  const auto next = [&](int x) -> int32_t {
    const int64_t k = pos[x]++;
    const int64_t nf = fc[x + 1] - fc[x];
    return (int32_t)(k < nf ? fc[x] + k : n_full + sc[x] + (k - nf));
  };
  for (int64_t i = 0; i < n_waves; ++i) S->tile_order[(size_t)i] = next((int)((i / kWaves) % kClaimCounters));
  for (int64_t i = n_waves; i < n; ++i) S->tile_order[(size_t)i] = next((int)((i - n_waves) % kClaimCounters));
  // A permutation of the tiles, or the kernel would skip or repeat one.
  std::vector<uint8_t> seen((size_t)n, 0);
  for (int64_t i = 0; i < n; ++i) {
    const int32_t t = S->tile_order[(size_t)i];
    if (t < 0 || t >= n || seen[(size_t)t]) return "tile order is not a permutation";
    seen[(size_t)t] = 1;
  }
  return "";
}

}  // namespace

extern "C" {

mist_status mist_space_create(const mist_model_desc* m, const mist_hw_desc* hw, int32_t n_hw,
                              const mist_space_desc* s, const mist_allocator* alloc, mist_space** out) {
  if (!out) return fail(MIST_E_INVALID, "out is null");
  *out = nullptr;
  try {
    const std::string why = validate(m, hw, n_hw, s);
    if (!why.empty()) return fail(MIST_E_INVALID, why);
    if (alloc && (!alloc->alloc || !alloc->free)) return fail(MIST_E_INVALID, "allocator callbacks missing");
    mist_space* S = new (std::nothrow) mist_space();
    if (!S) return fail(MIST_E_NOMEM, "host allocation failed");
    S->model = *m;
    S->hw.assign(hw, hw + n_hw);
    S->D = s->n_devices;
    S->B = s->global_batch;
    S->mb.assign(s->mb, s->mb + s->n_mb);
    S->R = s->n_ratios;
    S->NB = s->n_buckets;
    S->l_rule = s->l_rule;
    S->ratio_om.assign(s->ratios, s->ratios + s->n_ratios);
    for (int32_t i = 0; i < s->n_ratios; ++i) S->ratio_om.push_back(1.0 - s->ratios[i]);
    S->tile_configs = s->tile_configs > 0 ? s->tile_configs : kMinTileConfigs;
    S->max_blocks = s->max_blocks;
    S->cand_window = s->cand_window;
    S->A = s->n_alphas;
    S->alphas.assign(s->alphas, s->alphas + s->n_alphas);
    for (int32_t i = 0; i < s->n_alphas; ++i) S->betas.push_back(1.0 - s->alphas[i]);
    if (alloc) {
      S->alloc = *alloc;
      S->custom_alloc = true;
    }
    mist_status ecode = MIST_E_INVALID;
    const std::string err = enumerate(S, &ecode);
    if (!err.empty()) {
      delete S;
      return fail(ecode, err);
    }
    mist_status rc = MIST_OK;
    // Persistent evaluation grid: as many blocks as fit on the device at once.
    int64_t resident_blocks = 1;
    {
      int dev = 0, cus = 0;
      hipError_t e = hipGetDevice(&dev);
      if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
      if (e != hipSuccess) rc = fail_hip(e, "device attributes");
      const int per_cu = eval_blocks_per_cu(S->R, S->A > 0 ? kModeAlpha : kModeBuckets);
      resident_blocks = std::max<int64_t>(1, (int64_t)cus * (per_cu > 0 ? per_cu : 1));
      if (S->max_blocks > 0) resident_blocks = std::min<int64_t>(resident_blocks, S->max_blocks);
      S->cus = cus;
      S->device = dev;
    }
    if (!rc) {
      const std::string terr = build_tiles(S, resident_blocks * kWaves);
      if (!terr.empty()) rc = fail(MIST_E_INVALID, terr);
    }
    if (!rc) {
      const int64_t waves_needed = (int64_t)(S->tiles.size() + kWaves - 1) / kWaves;
      S->eval_grid = (int32_t)std::max<int64_t>(1, std::min<int64_t>(resident_blocks, waves_needed));
      int32_t n_full = 0;
      for (const DevGroup& G : S->groups) {
        S->max_group_tiles = std::max(S->max_group_tiles, G.n_tiles + G.n_tail);
        n_full += G.n_tiles;
      }
      const std::string oerr = build_tile_order(S, (int64_t)S->eval_grid * kWaves, n_full);
      if (!oerr.empty()) rc = fail(MIST_E_INVALID, oerr);
    }
    if (!rc) rc = upload(S, &S->d_groups, S->groups, "groups");
    if (!rc) rc = upload(S, &S->d_pairs, S->pairs, "pairs");
    if (!rc) rc = upload(S, &S->d_tiles, S->tiles, "tiles");
    if (!rc) rc = upload(S, &S->d_tile_order, S->tile_order, "tile order");
    if (!rc) rc = upload(S, &S->d_hws, S->hws, "hardware tables");
    if (!rc) rc = upload(S, &S->d_ratio, S->ratio_om, "ratios");
    if (!rc) rc = upload(S, &S->d_pk_group, S->pk_group, "pair groups");
    if (!rc && S->A > 0) rc = upload(S, &S->d_alpha, S->alphas, "weight samples");
    if (!rc && S->A > 0) rc = upload(S, &S->d_beta, S->betas, "weight samples");
    if (!rc) {
      S->d_pk = (PairK*)dev_alloc(S, S->pk_group.size() * sizeof(PairK), nullptr);
      S->d_work = (int32_t*)dev_alloc(S, sizeof(int32_t) * kClaimCounters * kCounterStride, nullptr);
      if (!S->d_pk || !S->d_work) rc = fail(MIST_E_NOMEM, "device allocation failed: pair constants");
    }
    const size_t nt = S->tiles.size(), ng = S->groups.size();
    if (!rc) {
      S->d_part_obj = (double*)dev_alloc(S, nt * 64 * sizeof(double), nullptr);
      S->d_part_id = (uint64_t*)dev_alloc(S, nt * 64 * sizeof(uint64_t), nullptr);
      S->d_bucket_obj = (double*)dev_alloc(S, ng * 64 * sizeof(double), nullptr);
      S->d_bucket_id = (uint64_t*)dev_alloc(S, ng * 64 * sizeof(uint64_t), nullptr);
      S->d_best_obj = (double*)dev_alloc(S, ng * sizeof(double), nullptr);
      S->d_best_id = (uint64_t*)dev_alloc(S, ng * sizeof(uint64_t), nullptr);
      S->d_frontier = (uint64_t*)dev_alloc(S, ng * sizeof(uint64_t), nullptr);
      if (!S->d_part_obj || !S->d_part_id || !S->d_bucket_obj || !S->d_bucket_id || !S->d_best_obj ||
          !S->d_best_id || !S->d_frontier)
        rc = fail(MIST_E_NOMEM, "device allocation failed: results");
    }
    if (!rc && S->A > 0) {
      const size_t A = (size_t)S->A;
      S->d_part_aobj = (double*)dev_alloc(S, nt * A * sizeof(double), nullptr);
      S->d_part_aid = (uint64_t*)dev_alloc(S, nt * A * sizeof(uint64_t), nullptr);
      S->d_alpha_obj = (double*)dev_alloc(S, ng * A * sizeof(double), nullptr);
      S->d_alpha_id = (uint64_t*)dev_alloc(S, ng * A * sizeof(uint64_t), nullptr);
      if (!S->d_part_aobj || !S->d_part_aid || !S->d_alpha_obj || !S->d_alpha_id)
        rc = fail(MIST_E_NOMEM, "device allocation failed: weight-sample results");
    }
    if (!rc) {
      // The buffers came from the null stream's blocks (mist_allocator): work queued there
      // before them finishes before any later call uses them on another stream.
      const hipError_t e = hipStreamSynchronize(nullptr);
      if (e != hipSuccess) rc = fail_hip(e, "hipStreamSynchronize");
    }
    if (rc) {
      dev_free_all(S);
      delete S;
      return rc;
    }
    *out = S;
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(MIST_E_INVALID, "unexpected error");
  }
}

mist_status mist_eval_space(mist_space* S, void* hip_stream) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  hipStream_t st = (hipStream_t)hip_stream;
  // Work of this space still queued on another stream uses the same buffers and tile
  // counters: it finishes first.
  if (S->evaluated && S->stream != st) {
    const hipError_t e = hipStreamSynchronize(S->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  }
  if (S->exact_launched && S->exact_stream != st) {
    const hipError_t e = hipStreamSynchronize(S->exact_stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  }
  const EvalArgs ea = eval_args(S);
  int rc = launch_pairs(ea, st);
  if (rc) return fail_hip((hipError_t)rc, "pair kernel launch");
  hipEvent_t* ev = nullptr;
  if (S->timing) {
    while (S->events.size() < S->events_used + 3) {
      hipEvent_t e;
      const hipError_t rc = hipEventCreate(&e);
      if (rc != hipSuccess) return fail_hip(rc, "hipEventCreate");
      S->events.push_back(e);
    }
    ev = &S->events[S->events_used];
    S->events_used += 3;
    const hipError_t e = hipEventRecord(ev[0], st);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
  }
  rc = launch_eval(ea, S->eval_grid, S->A > 0 ? kModeAlpha : kModeBuckets, st);
  if (rc) return fail_hip((hipError_t)rc, "evaluation kernel launch");
  if (ev) {
    const hipError_t e = hipEventRecord(ev[1], st);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
  }
  ReduceArgs r{};
  r.groups = S->d_groups;
  r.n_groups = (int64_t)S->groups.size();
  r.NB = S->NB;
  r.max_group_tiles = S->max_group_tiles;
  r.part_obj = S->d_part_obj;
  r.part_id = S->d_part_id;
  r.bucket_obj = S->d_bucket_obj;
  r.bucket_id = S->d_bucket_id;
  r.best_obj = S->d_best_obj;
  r.best_id = S->d_best_id;
  r.frontier = S->d_frontier;
  r.n_alpha = S->A;
  r.part_aobj = S->d_part_aobj;
  r.part_aid = S->d_part_aid;
  r.alpha_obj = S->d_alpha_obj;
  r.alpha_id = S->d_alpha_id;
  rc = launch_reduce(r, st);
  if (rc) return fail_hip((hipError_t)rc, "reduction kernel launch");
  if (ev) {
    const hipError_t e = hipEventRecord(ev[2], st);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
  }
  S->evaluated = true;
  S->stream = st;
  S->exact_done = false;
  return MIST_OK;
}

// Grid of the persistent evaluation kernel in a given variant.
static int32_t mode_grid(const mist_space* S, int mode) {
  const int per_cu = eval_blocks_per_cu(S->R, mode);
  int64_t resident = std::max<int64_t>(1, (int64_t)S->cus * (per_cu > 0 ? per_cu : 1));
  if (S->max_blocks > 0) resident = std::min<int64_t>(resident, S->max_blocks);
  const int64_t waves_needed = (int64_t)(S->tiles.size() + kWaves - 1) / kWaves;
  return (int32_t)std::max<int64_t>(1, std::min<int64_t>(resident, waves_needed));
}

mist_status mist_eval_pareto_exact(mist_space* S, void* hip_stream) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  mist_status rc = wait_results(S);
  if (rc) return rc;
  try {
    hipStream_t st = (hipStream_t)hip_stream;
    const size_t nt = S->tiles.size(), ng = S->groups.size();
    // The host offset tables below are uploaded asynchronously: a previous call on another
    // stream must be done with them before they are rewritten.
    if (S->exact_launched && S->exact_stream != st) {
      const hipError_t e = hipStreamSynchronize(S->exact_stream);
      if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    }
    S->exact_done = false;
    if (!S->d_filt) {
      // Windows: ceil(configurations / div) slots per tile.
      const int64_t R2 = (int64_t)S->R * S->R;
      auto slots = [&](int64_t div) {
        int64_t n = 0;
        for (const DevTile& T : S->tiles) n += ((int64_t)(T.strip_end - T.strip_begin) * R2 + div - 1) / div;
        return n;
      };
      int64_t div = S->cand_window > 0 ? S->cand_window : kWindowDiv;
      if (S->cand_window == 0)
        while (slots(div) > kWindowSlots) div *= 2;
      S->h_slab_begin.assign(nt + 1, 0);
      for (size_t t = 0; t < nt; ++t) {
        const DevTile& T = S->tiles[t];
        S->h_slab_begin[t + 1] = S->h_slab_begin[t] + ((int64_t)(T.strip_end - T.strip_begin) * R2 + div - 1) / div;
      }
      const size_t n_slab = (size_t)std::max<int64_t>(S->h_slab_begin[nt], 1);
      S->d_filt = (FiltEntry*)dev_alloc(S, std::max<size_t>(ng, 1) * 64 * sizeof(FiltEntry), st);
      S->d_cnt_tile = (int32_t*)dev_alloc(S, std::max<size_t>(nt, 1) * sizeof(int32_t), st);
      S->d_tile_off = (int64_t*)dev_alloc(S, std::max<size_t>(nt, 1) * sizeof(int64_t), st);
      S->d_tile_end = (int64_t*)dev_alloc(S, std::max<size_t>(nt, 1) * sizeof(int64_t), st);
      S->d_list = (int32_t*)dev_alloc(S, std::max<size_t>(nt, 1) * sizeof(int32_t), st);
      S->d_live = (uint8_t*)dev_alloc(S, std::max<size_t>(nt, 1), st);
      S->d_seg = (int64_t*)dev_alloc(S, (ng + 1) * sizeof(int64_t), st);
      S->d_seg_end = (int64_t*)dev_alloc(S, std::max<size_t>(ng, 1) * sizeof(int64_t), st);
      S->d_front_cnt = (int64_t*)dev_alloc(S, std::max<size_t>(ng, 1) * sizeof(int64_t), st);
      S->d_slab_begin = (int64_t*)dev_alloc(S, (nt + 1) * sizeof(int64_t), st);
      S->d_slab_key = (uint64_t*)dev_alloc(S, n_slab * 8, st);
      S->d_slab_obj = (double*)dev_alloc(S, n_slab * 8, st);
      S->d_slab_id = (uint64_t*)dev_alloc(S, n_slab * 8, st);
      // The pool holds as many slots as all windows together (at most kPoolSlots): the windows
      // of tiles that hold no candidate stay empty, so the overflow of the others can be large.
      S->pool_cap = std::min<int64_t>(kPoolSlots, std::max<int64_t>((int64_t)n_slab, 1));
      const size_t n_pool = (size_t)S->pool_cap;
      S->d_pool_count = (unsigned long long*)dev_alloc(S, 256, st);
      S->d_pool_key = (uint64_t*)dev_alloc(S, n_pool * 8, st);
      S->d_pool_obj = (double*)dev_alloc(S, n_pool * 8, st);
      S->d_pool_id = (uint64_t*)dev_alloc(S, n_pool * 8, st);
      S->d_pool_tile = (int32_t*)dev_alloc(S, n_pool * 4, st);
      S->d_pool_rank = (int32_t*)dev_alloc(S, n_pool * 4, st);
      S->d_tile_drop = (uint8_t*)dev_alloc(S, std::max<size_t>(nt, 1), st);
      {
        const size_t bytes = 8 * (2 * nt + ng + 1) + 4 * (2 * nt) + 64 + 8 + nt;
        void* p = nullptr;
        if (hipHostMalloc(&p, bytes, hipHostMallocDefault) != hipSuccess) p = nullptr;
        S->h_pinned = p;
        if (p) {
          char* q = (char*)p;
          S->h_tile_off = (int64_t*)q;
          S->h_tile_end = S->h_tile_off + nt;
          S->h_seg = S->h_tile_end + nt;
          S->h_cnt = (int32_t*)(S->h_seg + ng + 1);
          S->h_list = S->h_cnt + nt;
          S->h_pool_count = (unsigned long long*)(S->h_list + nt + 16);  // 8-byte aligned: nt ints + 64 B
          S->h_drop = (uint8_t*)(S->h_pool_count + 1);
        }
      }
      void** bufs[] = {(void**)&S->d_filt,      (void**)&S->d_cnt_tile,   (void**)&S->d_tile_off,
                       (void**)&S->d_tile_end,  (void**)&S->d_list,       (void**)&S->d_seg, (void**)&S->d_seg_end, (void**)&S->d_live,
                       (void**)&S->d_front_cnt, (void**)&S->d_slab_begin, (void**)&S->d_slab_key,
                       (void**)&S->d_slab_obj,  (void**)&S->d_slab_id,    (void**)&S->d_pool_count,
                       (void**)&S->d_pool_key,  (void**)&S->d_pool_obj,   (void**)&S->d_pool_id,
                       (void**)&S->d_pool_tile, (void**)&S->d_pool_rank,  (void**)&S->d_tile_drop};
      bool ok = S->h_pinned != nullptr;
      for (void** b : bufs) ok = ok && *b;
      if (!ok) {  // free what was allocated: the next call starts over
        for (void** b : bufs) {
          dev_free_one(S, *b);
          *b = nullptr;
        }
        if (S->h_pinned) (void)hipHostFree(S->h_pinned);
        S->h_pinned = nullptr;
        return fail(MIST_E_NOMEM, "device allocation failed: exact frontier");
      }
      const hipError_t e = copy_sync(S->d_slab_begin, S->h_slab_begin.data(), (nt + 1) * sizeof(int64_t),
                                     hipMemcpyHostToDevice);
      if (e != hipSuccess) return fail_hip(e, "exact frontier: windows");
    }
    // Pass 1: every tile writes its candidates to its window and counts them.
    EvalArgs ea = eval_args(S);
    ea.filt = S->d_filt;
    ea.cnt_tile = S->d_cnt_tile;
    ea.win_begin = S->d_slab_begin;
    ea.win_end = S->d_slab_begin + 1;
    ea.tile_list = nullptr;
    ea.n_list = 0;
    ea.tile_live = S->d_live;
    ea.cand_key = S->d_slab_key;
    ea.cand_obj = S->d_slab_obj;
    ea.cand_id = S->d_slab_id;
    ea.pool_count = S->d_pool_count;
    ea.pool_cap = S->pool_cap;
    ea.pool_key = S->d_pool_key;
    ea.pool_obj = S->d_pool_obj;
    ea.pool_id = S->d_pool_id;
    ea.pool_tile = S->d_pool_tile;
    ea.pool_rank = S->d_pool_rank;
    ea.tile_drop = S->d_tile_drop;
    int k = launch_filter(ea, S->d_bucket_obj, S->d_bucket_id, S->d_filt, st);
    if (!k) k = launch_live(ea, S->d_filt, S->d_live, st);
    if (!k) k = launch_pairs(ea, st);  // also resets the tile counters and the pool
    if (!k) k = launch_eval(ea, mode_grid(S, kModeEmit), kModeEmit, st);
    if (k) return fail_hip((hipError_t)k, "exact frontier: candidates");
    hipError_t e = copy_async(S->h_cnt, S->d_cnt_tile, nt * sizeof(int32_t), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = copy_async(S->h_drop, S->d_tile_drop, nt, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = copy_async(S->h_pool_count, S->d_pool_count, 8, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(e, "exact frontier: counts");
    // The pool counter is cleared by the pair-constants kernel.  A space without pairs has no
    // tile: neither that kernel nor the candidate pass runs, the counter keeps whatever its
    // block held, and the pool is empty.
    const int64_t n_pool = ea.n_pk > 0 ? std::min<int64_t>((int64_t)*S->h_pool_count, S->pool_cap) : 0;
    // Candidate slots in group order: a group's full-size tiles, then its small ones.  Tiles with
    // a candidate that found no place (its window and the pool full) are listed for pass 2.
    S->n_list = 0;
    int64_t off = 0;
    for (size_t t = 0; t < nt; ++t)
      if (S->h_cnt[t] == INT32_MAX) return fail(MIST_E_RANGE, "exact frontier: 2^31 or more candidates in a tile");
    auto place = [&](int32_t t) {
      S->h_tile_off[t] = off;
      off += S->h_cnt[t];
      S->h_tile_end[t] = off;
      if (S->h_drop[t]) S->h_list[S->n_list++] = t;
    };
    for (size_t g = 0; g < ng; ++g) {
      const DevGroup& G = S->groups[g];
      S->h_seg[g] = off;
      for (int32_t t = G.tile_begin; t < G.tile_begin + G.n_tiles; ++t) place(t);
      for (int32_t t = G.tail_begin; t < G.tail_begin + G.n_tail; ++t) place(t);
    }
    S->h_seg[ng] = off;
    if (off >= ((int64_t)1 << 32)) return fail(MIST_E_RANGE, "exact frontier: more than 2^32 candidates");
    if (off > S->cand_cap) {
      void* old[] = {S->d_cand_key, S->d_cand_id, S->d_key_sorted, S->d_cand_obj, S->d_idx_in, S->d_idx_out,
                     S->d_front_key, S->d_front_id, S->d_front_obj};
      for (void* p : old) dev_free_one(S, p);
      const size_t n = (size_t)off;
      S->d_cand_key = (uint64_t*)dev_alloc(S, n * 8, st);
      S->d_cand_id = (uint64_t*)dev_alloc(S, n * 8, st);
      S->d_key_sorted = (uint64_t*)dev_alloc(S, n * 8, st);
      S->d_cand_obj = (double*)dev_alloc(S, n * 8, st);
      S->d_idx_in = (uint32_t*)dev_alloc(S, n * 4, st);
      S->d_idx_out = (uint32_t*)dev_alloc(S, n * 4, st);
      S->d_front_key = (uint64_t*)dev_alloc(S, n * 8, st);
      S->d_front_id = (uint64_t*)dev_alloc(S, n * 8, st);
      S->d_front_obj = (double*)dev_alloc(S, n * 8, st);
      S->cand_cap = off;
      if (!S->d_cand_key || !S->d_cand_id || !S->d_key_sorted || !S->d_cand_obj || !S->d_idx_in ||
          !S->d_idx_out || !S->d_front_key || !S->d_front_id || !S->d_front_obj) {
        S->cand_cap = 0;
        return fail(MIST_E_NOMEM, "device allocation failed: exact frontier candidates");
      }
    }
    const int32_t n_list = S->n_list;
    S->exact_launched = true;
    S->exact_stream = st;
    e = copy_async(S->d_tile_off, S->h_tile_off, nt * sizeof(int64_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess)
      e = copy_async(S->d_seg, S->h_seg, (ng + 1) * sizeof(int64_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess && n_list > 0)
      e = copy_async(S->d_tile_end, S->h_tile_end, nt * sizeof(int64_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess && n_list > 0)
      e = copy_async(S->d_list, S->h_list, (size_t)n_list * sizeof(int32_t), hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return fail_hip(e, "exact frontier: offsets");
    // The windows that held their tile's candidates move to group order; pass 2 evaluates the
    // listed tiles again, writing straight to their slots.
    k = launch_compact(S->d_slab_key, S->d_slab_obj, S->d_slab_id, S->d_slab_begin, S->d_cnt_tile, S->d_tile_drop,
                       S->d_tile_off, (int32_t)nt, S->d_cand_key, S->d_cand_obj, S->d_cand_id, st);
    if (!k)
      k = launch_pool_place(S->d_pool_key, S->d_pool_obj, S->d_pool_id, S->d_pool_tile, S->d_pool_rank, n_pool,
                            S->d_tile_drop, S->d_tile_off, S->d_cand_key, S->d_cand_obj, S->d_cand_id, st);
    if (!k && n_list > 0) {
      ea.pool_count = nullptr;  // exact slots: nothing overflows
      ea.tile_drop = nullptr;
      ea.win_begin = S->d_tile_off;
      ea.win_end = S->d_tile_end;
      ea.tile_list = S->d_list;
      ea.n_list = n_list;
      ea.cand_key = S->d_cand_key;
      ea.cand_obj = S->d_cand_obj;
      ea.cand_id = S->d_cand_id;
      k = launch_pairs(ea, st);
      if (!k) k = launch_eval(ea, mode_grid(S, kModeEmit), kModeEmit, st);
    }
    if (!k) k = launch_prefilter(S->d_cand_key, S->d_cand_obj, S->d_cand_id, S->d_seg, (int64_t)ng, S->d_seg_end, st);
    // The frontier's key array and the slot array d_idx_in serve as the sort's scratch (the scan
    // writes the frontier after the sort).
    if (!k)
      k = exact_sort(S->d_cand_key, S->d_key_sorted, S->d_idx_out, S->d_front_key, S->d_idx_in, (int64_t)ng,
                     S->d_seg, S->d_seg_end, st);
    if (!k)
      k = launch_front_scan(S->d_idx_out, S->d_key_sorted, S->d_cand_obj, S->d_cand_id, S->d_seg, S->d_seg_end,
                            (int64_t)ng, S->d_front_key, S->d_front_obj, S->d_front_id, S->d_front_cnt, st);
    if (k) return fail_hip((hipError_t)k, "exact frontier");
    S->n_cand = off;
    S->n_rerun = n_list;
    S->n_pooled = n_pool;
    S->exact_done = true;
    S->exact_stream = st;
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_exact_info(mist_space* S, int64_t* n_candidates, int64_t* n_kept, int32_t* n_tiles_live,
                            int32_t* n_tiles_again) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (!S->exact_done) return fail(MIST_E_STATE, "mist_eval_pareto_exact has not been called");
  hipError_t e = hipStreamSynchronize(S->exact_stream);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  try {
    const size_t ng = S->groups.size();
    std::vector<int64_t> ends(ng);
    e = copy_sync(ends.data(), S->d_seg_end, ng * sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy segment ends");
    int64_t kept = 0;
    for (size_t g = 0; g < ng; ++g) kept += ends[g] - S->h_seg[g];
    const size_t nt = S->tiles.size();
    std::vector<uint8_t> live(nt);
    e = copy_sync(live.data(), S->d_live, nt, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy live tiles");
    int32_t n_live = 0;
    for (uint8_t v : live) n_live += v ? 1 : 0;
    if (n_candidates) *n_candidates = S->n_cand;
    if (n_kept) *n_kept = kept;
    if (n_tiles_live) *n_tiles_live = n_live;
    if (n_tiles_again) *n_tiles_again = S->n_rerun;
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_exact_group_sizes(mist_space* S, int64_t g0, int64_t n, int64_t* candidates, int64_t* kept) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (!S->exact_done) return fail(MIST_E_STATE, "mist_eval_pareto_exact has not been called");
  if (g0 < 0 || n < 0 || g0 + n > (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group range");
  if (n == 0) return MIST_OK;
  try {
    std::vector<int64_t> seg((size_t)n + 1), end((size_t)n);
    hipError_t e = hipStreamSynchronize(S->exact_stream);
    if (e == hipSuccess) e = copy_sync(seg.data(), S->d_seg + g0, ((size_t)n + 1) * sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = copy_sync(end.data(), S->d_seg_end + g0, (size_t)n * sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "exact frontier: group sizes");
    for (int64_t i = 0; i < n; ++i) {
      if (candidates) candidates[i] = seg[(size_t)i + 1] - seg[(size_t)i];
      if (kept) kept[i] = end[(size_t)i] - seg[(size_t)i];
    }
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_get_pareto_exact(mist_space* S, int64_t g, mist_result* out, int64_t cap, int64_t* n_out) {
  if (!S || !n_out || (!out && cap > 0)) return fail(MIST_E_INVALID, "null argument");
  if (!S->exact_done) return fail(MIST_E_STATE, "mist_eval_pareto_exact has not been called");
  if (g < 0 || g >= (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group out of range");
  hipError_t e = hipStreamSynchronize(S->exact_stream);
  if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  try {
    int64_t n = 0;
    e = copy_sync(&n, S->d_front_cnt + g, sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy frontier count");
    *n_out = n;
    if (n > cap) return fail(MIST_E_RANGE, "cap is smaller than the frontier");
    if (n == 0) return MIST_OK;
    const size_t b = (size_t)S->h_seg[g];
    std::vector<uint64_t> keys(n), ids(n);
    std::vector<double> objs(n);
    e = copy_sync(keys.data(), S->d_front_key + b, n * 8, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = copy_sync(ids.data(), S->d_front_id + b, n * 8, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = copy_sync(objs.data(), S->d_front_obj + b, n * 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy frontier");
    mist_status rc = fill_results(S, ids.data(), objs.data(), n, out);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i) {
      double mem;
      std::memcpy(&mem, &keys[i], 8);
      if (mem != out[i].mem) return fail(MIST_E_DEVICE, "re-evaluated memory differs");
    }
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_get_best(mist_space* S, int64_t g0, int64_t n, mist_result* out) {
  if (!S || (!out && n > 0)) return fail(MIST_E_INVALID, "null argument");
  if (g0 < 0 || n < 0 || g0 + n > (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group range");
  mist_status rc = wait_results(S);
  if (rc) return rc;
  if (n == 0) return MIST_OK;
  try {
    std::vector<uint64_t> ids(n);
    std::vector<double> objs(n);
    hipError_t e = copy_sync(ids.data(), S->d_best_id + g0, n * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      e = copy_sync(objs.data(), S->d_best_obj + g0, n * sizeof(double), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy best");
    return fill_results(S, ids.data(), objs.data(), n, out);
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_get_alpha(mist_space* S, int64_t g0, int64_t n, mist_result* out) {
  if (!S || (!out && n > 0)) return fail(MIST_E_INVALID, "null argument");
  if (S->A == 0) return fail(MIST_E_STATE, "the space has no weight samples");
  if (g0 < 0 || n < 0 || g0 + n > (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group range");
  mist_status rc = wait_results(S);
  if (rc) return rc;
  if (n == 0) return MIST_OK;
  try {
    const size_t A = (size_t)S->A, m = (size_t)n * A;
    std::vector<uint64_t> ids(m);
    std::vector<double> objs(m);
    hipError_t e = copy_sync(ids.data(), S->d_alpha_id + (size_t)g0 * A, m * sizeof(uint64_t),
                             hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      e = copy_sync(objs.data(), S->d_alpha_obj + (size_t)g0 * A, m * sizeof(double), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy weight-sample results");
    std::vector<uint64_t> want;
    for (size_t i = 0; i < m; ++i)
      if (ids[i] != MIST_NONE) want.push_back(ids[i]);
    std::vector<double> vals(want.size() * 4);
    rc = eval_ids_impl(S, want.data(), (int64_t)want.size(), vals.data(), S->stream);
    if (rc) return rc;
    size_t w = 0;
    for (size_t i = 0; i < m; ++i) {
      mist_result& r = out[i];
      std::memset(&r, 0, sizeof(r));
      r.id = ids[i];
      r.obj = objs[i];
      if (ids[i] == MIST_NONE) {
        r.t = r.d = r.mem = std::numeric_limits<double>::infinity();
        r.bucket = -1;
        r.cfg.hw = -1;
        continue;
      }
      r.t = vals[4 * w + 0];
      r.d = vals[4 * w + 1];
      r.mem = vals[4 * w + 2];
      ++w;
      decode_host(S, r.id, &r.cfg);
      const size_t a = i % A;
      const double v = std::fma(S->alphas[a] * (double)r.cfg.G, r.t, S->betas[a] * r.d);
      if (v != r.obj) return fail(MIST_E_DEVICE, "re-evaluated weighted objective differs");
      r.bucket = bucket_host(S, S->hws[r.cfg.hw], r.mem);
    }
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_plan_pipeline(mist_space* S, int32_t hw, int32_t pp, mist_plan* out) {
  if (!S || !out) return fail(MIST_E_INVALID, "null argument");
  if (hw < 0 || hw >= (int32_t)S->hw.size()) return fail(MIST_E_RANGE, "hardware sample out of range");
  if (pp < 0 || pp > MIST_MAX_STAGES) return fail(MIST_E_INVALID, "pp out of range");
  mist_status rc = wait_results(S);
  if (rc) return rc;
  try {
    const size_t A = (size_t)S->A, ng = S->groups.size();
    std::vector<uint64_t> best(ng), alpha(ng * A);
    hipError_t e = copy_sync(best.data(), S->d_best_id, ng * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e == hipSuccess && A)
      e = copy_sync(alpha.data(), S->d_alpha_id, ng * A * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy frontier points");
    std::vector<mist_stage_point> pts;
    std::vector<uint64_t> ids;
    for (size_t g = 0; g < ng; ++g) {
      if (S->groups[g].hw != hw || (pp != 0 && S->groups[g].PP != pp)) continue;
      std::vector<uint64_t> mine(1 + A);
      mine[0] = best[g];
      for (size_t a = 0; a < A; ++a) mine[1 + a] = alpha[g * A + a];
      std::sort(mine.begin(), mine.end());
      mine.erase(std::unique(mine.begin(), mine.end()), mine.end());
      const DevGroup& G = S->groups[g];
      for (uint64_t id : mine) {
        if (id == MIST_NONE) continue;
        mist_stage_point p{};
        p.G = G.G; p.PP = G.PP; p.k = G.k; p.l = G.l; p.id = id;
        pts.push_back(p);
        ids.push_back(id);
      }
    }
    std::vector<double> vals(ids.size() * 4);
    rc = eval_ids_impl(S, ids.data(), (int64_t)ids.size(), vals.data(), S->stream);
    if (rc) return rc;
    for (size_t i = 0; i < pts.size(); ++i) {
      pts[i].t = vals[4 * i + 0];
      pts[i].d = vals[4 * i + 1];
    }
    rc = mist_plan_points(pts.data(), (int64_t)pts.size(), S->model.n_layers, pp, out);
    if (rc) return rc;
    out->hw = hw;
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_get_buckets(mist_space* S, int64_t g0, int64_t n, uint64_t* ids, double* objs,
                             uint64_t* masks) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (g0 < 0 || n < 0 || g0 + n > (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group range");
  mist_status rc = wait_results(S);
  if (rc) return rc;
  if (n == 0) return MIST_OK;
  try {
    const int NB = S->NB;
    std::vector<uint64_t> bid((size_t)n * 64);
    std::vector<double> bobj((size_t)n * 64);
    hipError_t e = copy_sync(bid.data(), S->d_bucket_id + g0 * 64, bid.size() * sizeof(uint64_t),
                             hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      e = copy_sync(bobj.data(), S->d_bucket_obj + g0 * 64, bobj.size() * sizeof(double),
                    hipMemcpyDeviceToHost);
    if (e == hipSuccess && masks)
      e = copy_sync(masks, S->d_frontier + g0, n * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy buckets");
    for (int64_t i = 0; i < n; ++i)
      for (int j = 0; j < NB; ++j) {
        if (ids) ids[i * NB + j] = bid[i * 64 + j];
        if (objs) objs[i * NB + j] = bobj[i * 64 + j];
      }
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_get_pareto(mist_space* S, int64_t g, mist_result* out, int32_t cap, int32_t* n_out) {
  if (!S || !n_out) return fail(MIST_E_INVALID, "null argument");
  if (g < 0 || g >= (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group index");
  const int NB = S->NB;
  std::vector<uint64_t> ids(NB);
  std::vector<double> objs(NB);
  uint64_t mask = 0;
  mist_status rc = mist_get_buckets(S, g, 1, ids.data(), objs.data(), &mask);
  if (rc) return rc;
  std::vector<uint64_t> fid;
  std::vector<double> fobj;
  for (int j = 0; j < NB; ++j)
    if (mask >> j & 1) {
      fid.push_back(ids[j]);
      fobj.push_back(objs[j]);
    }
  *n_out = (int32_t)fid.size();
  if ((int32_t)fid.size() > cap) return fail(MIST_E_RANGE, "output capacity too small");
  if (fid.empty()) return MIST_OK;
  if (!out) return fail(MIST_E_INVALID, "out is null");
  return fill_results(S, fid.data(), fobj.data(), (int64_t)fid.size(), out);
}

mist_status mist_space_info(const mist_space* S, uint64_t* n_configs, int64_t* n_groups, int32_t* n_buckets) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (n_configs) *n_configs = S->n_configs;
  if (n_groups) *n_groups = (int64_t)S->groups.size();
  if (n_buckets) *n_buckets = S->NB;
  return MIST_OK;
}

mist_status mist_get_group_key(const mist_space* S, int64_t g, mist_group_key* out) {
  if (!S || !out) return fail(MIST_E_INVALID, "null argument");
  if (g < 0 || g >= (int64_t)S->groups.size()) return fail(MIST_E_RANGE, "group index");
  const DevGroup& d = S->groups[g];
  out->hw = d.hw; out->G = d.G; out->PP = d.PP; out->k = d.k; out->l = d.l; out->n_pairs = d.n_pairs;
  out->base = d.base;
  out->size = (uint64_t)d.n_pairs * (uint64_t)(d.l + 1) * 4ull * (uint64_t)S->R * S->R * S->R * S->R;
  return MIST_OK;
}

mist_status mist_decode(const mist_space* S, uint64_t id, mist_config* out) {
  if (!S || !out) return fail(MIST_E_INVALID, "null argument");
  if (id >= S->n_configs) return fail(MIST_E_RANGE, "id out of range");
  decode_host(S, id, out);
  return MIST_OK;
}

mist_status mist_eval_ids(mist_space* S, const uint64_t* ids, int64_t n, double* out, void* hip_stream) {
  if (!S || ((!ids || !out) && n > 0) || n < 0) return fail(MIST_E_INVALID, "null argument");
  try {
    return eval_ids_impl(S, ids, n, out, (hipStream_t)hip_stream);
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_eval_ids_noalloc(mist_space* S, const uint64_t* ids, int64_t n, double* out, void* hip_stream) {
  if (!S || ((!ids || !out) && n > 0) || n < 0) return fail(MIST_E_INVALID, "null argument");
  if (n > kNoAllocMaxIds)
    return fail(MIST_E_RANGE, "mist_eval_ids_noalloc: at most " + std::to_string(kNoAllocMaxIds) +
                                  " ids per call (a fixed 4 MiB device scratch)");
  if (n == 0) return MIST_OK;
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] >= S->n_configs) return fail(MIST_E_RANGE, "id out of range");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  if (dev != S->device) return fail(MIST_E_INVALID, "the space's device must be the current device");
  void* scratch = nullptr;
  const int rc = noalloc_scratch(&scratch);
  if (rc) return fail_hip((hipError_t)rc, "device scratch address");
  // Layout: ids [n] uint64, then results [n][4] doubles (8-byte aligned).  Both are written in
  // full before they are read, so nothing needs clearing.
  uint64_t* d_ids = (uint64_t*)scratch;
  double* d_out = (double*)((char*)scratch + (size_t)n * sizeof(uint64_t));
  hipStream_t st = (hipStream_t)hip_stream;
  e = copy_async(d_ids, ids, (size_t)n * sizeof(uint64_t), hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return fail_hip(e, "hipMemcpyAsync ids");
  const int k = launch_eval_ids(eval_args(S), d_ids, n, d_out, st);
  if (k) {
    (void)hipStreamSynchronize(st);
    return fail_hip((hipError_t)k, "eval_ids launch");
  }
  e = copy_async(out, d_out, (size_t)n * 4 * sizeof(double), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail_hip(e, "mist_eval_ids_noalloc results");
  return MIST_OK;
}

mist_status mist_set_timing(mist_space* S, int32_t on) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (S->evaluated) {
    const hipError_t e = hipStreamSynchronize(S->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  }
  S->timing = on != 0;
  S->events_used = 0;
  return MIST_OK;
}

mist_status mist_read_timing(mist_space* S, double* eval_ms, double* reduce_ms, int64_t* n_evals) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (!S->timing) return fail(MIST_E_STATE, "timing is off");
  double a = 0.0, b = 0.0;
  const size_t n = S->events_used / 3;
  if (n) {
    const hipError_t e = hipEventSynchronize(S->events[S->events_used - 1]);
    if (e != hipSuccess) return fail_hip(e, "hipEventSynchronize");
  }
  for (size_t i = 0; i < n; ++i) {
    float x = 0.f, y = 0.f;
    hipError_t e = hipEventElapsedTime(&x, S->events[3 * i], S->events[3 * i + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&y, S->events[3 * i + 1], S->events[3 * i + 2]);
    if (e != hipSuccess) return fail_hip(e, "hipEventElapsedTime");
    a += x;
    b += y;
  }
  S->events_used = 0;
  if (eval_ms) *eval_ms = a;
  if (reduce_ms) *reduce_ms = b;
  if (n_evals) *n_evals = (int64_t)n;
  return MIST_OK;
}

mist_status mist_tile_info(const mist_space* S, int32_t t, int64_t* group, uint64_t* first_id, int64_t* n_configs) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (t < 0 || (size_t)t >= S->tiles.size()) return fail(MIST_E_RANGE, "tile out of range");
  const DevTile& T = S->tiles[t];
  const uint64_t R2 = (uint64_t)S->R * (uint64_t)S->R;
  if (group) *group = T.group;
  if (first_id) *first_id = S->groups[T.group].base + (uint64_t)T.strip_begin * R2;
  if (n_configs) *n_configs = (int64_t)((uint64_t)(T.strip_end - T.strip_begin) * R2);
  return MIST_OK;
}

mist_status mist_debug_eval_tiles(mist_space* S, const int32_t* tiles, int32_t n, double* out, int64_t cap,
                                  void* hip_stream) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (n < 0 || (n > 0 && (!tiles || !out))) return fail(MIST_E_INVALID, "tiles and out must be given");
  if (n == 0) return MIST_OK;
  try {
    hipStream_t st = (hipStream_t)hip_stream;
    const int64_t R2 = (int64_t)S->R * S->R;
    std::vector<int64_t> off((size_t)n);
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
      if (tiles[i] < 0 || (size_t)tiles[i] >= S->tiles.size()) return fail(MIST_E_RANGE, "tile out of range");
      off[(size_t)i] = total;
      total += (int64_t)(S->tiles[tiles[i]].strip_end - S->tiles[tiles[i]].strip_begin) * R2;
    }
    if (total > cap) return fail(MIST_E_RANGE, "cap is smaller than the listed tiles' configurations");
    // Work of this space queued on other streams shares the tile counters: it finishes first.
    if (S->evaluated && S->stream != st) {
      const hipError_t e = hipStreamSynchronize(S->stream);
      if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    }
    if (S->exact_launched && S->exact_stream != st) {
      const hipError_t e = hipStreamSynchronize(S->exact_stream);
      if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    }
    TempBuf dlist(S, (size_t)n * sizeof(int32_t), st);
    TempBuf doff(S, (size_t)n * sizeof(int64_t), st);
    TempBuf dout(S, (size_t)std::max<int64_t>(total, 1) * kDumpWords * sizeof(double), st);
    if (!dlist.p || !doff.p || !dout.p) return fail(MIST_E_NOMEM, "device allocation failed: debug tiles");
    auto drained = [&](mist_status code) {
      (void)hipStreamSynchronize(st);
      return code;
    };
    hipError_t e = copy_async(dlist.p, tiles, (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = copy_async(doff.p, off.data(), (size_t)n * sizeof(int64_t), hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return drained(fail_hip(e, "debug tiles: upload"));
    EvalArgs ea = eval_args(S);
    ea.tile_list = (const int32_t*)dlist.p;
    ea.n_list = n;
    ea.dump = (double*)dout.p;
    ea.dump_off = (const int64_t*)doff.p;
    int k = launch_pairs(ea, st);  // pair constants, and the tile counters' reset
    if (!k) k = launch_eval(ea, mode_grid(S, kModeDump), kModeDump, st);
    if (k) return drained(fail_hip((hipError_t)k, "debug tiles: launch"));
    e = copy_async(out, dout.p, (size_t)total * kDumpWords * sizeof(double), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return drained(fail_hip(e, "debug tiles: results"));
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return fail(MIST_E_NOMEM, "host allocation failed");
  }
}

mist_status mist_launch_info(const mist_space* S, int64_t* n_tiles, int32_t* block, int32_t* strips_per_tile) {
  if (!S) return fail(MIST_E_INVALID, "space is null");
  if (n_tiles) *n_tiles = (int64_t)S->tiles.size();
  if (block) *block = kWaveTile;
  if (strips_per_tile) *strips_per_tile = S->strips_per_tile;
  return MIST_OK;
}

mist_status mist_space_destroy(mist_space* S) {
  if (!S) return MIST_OK;
  if (S->evaluated) (void)hipStreamSynchronize(S->stream);
  // The exact frontier may run on another stream; its buffers and host tables go below.
  if (S->exact_launched && S->exact_stream != S->stream) (void)hipStreamSynchronize(S->exact_stream);
  if (S->h_pinned) (void)hipHostFree(S->h_pinned);
  for (hipEvent_t e : S->events) (void)hipEventDestroy(e);
  dev_free_all(S);
  delete S;
  return MIST_OK;
}

const char* mist_last_error(void) { return g_error.c_str(); }

}  // extern "C"

namespace mist {
__attribute__((visibility("hidden"))) mist_status lib_fail(mist_status code, const std::string& msg) { return fail(code, msg); }
}  // namespace mist
