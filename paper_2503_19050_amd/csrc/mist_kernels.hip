// libmist kernels for gfx950: batched FP64 evaluation of Mist's per-stage cost model
// (Sec. 5.2-5.3, Eq. 4-6, Algorithm 1), feasibility filter, per-bucket and per-group
// reductions.
//
// Numerics: every floating-point operation of the cost model is an explicit IEEE binary64
// operation in a fixed order; the library is built with -ffp-contract=off and every fused
// multiply-add is an explicit __builtin_fma.  Reciprocals (1/F, 1/PCIe, 1/link, 1/DP,
// 1/eta(b), 1/phi) come from host divisions.  The results are therefore bit-reproducible
// and independent of the launch geometry.

#include <hip/hip_runtime.h>

#include "mist_internal.h"

namespace mist {
namespace {

constexpr uint64_t kNone = ~0ull;

__device__ __forceinline__ bool lex_less(double o1, uint64_t i1, double o2, uint64_t i2) {
  return o1 < o2 || (o1 == o2 && i1 < i2);
}

// ---------------------------------------------------------------------------------------
// Cost model, level by level.  Each level holds the quantities that depend on the digits
// fixed at that level: pair (b, TP, DP), recomputed layers c, ZeRO level z, then the
// weight, gradient, optimizer-state and activation offload ratios.
// ---------------------------------------------------------------------------------------
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

__device__ __forceinline__ PairK pair_level(const DevModel& m, int64_t PP, int64_t k, int64_t l,
                                            const DevPair& pr, const DevHw& hw) {
  const int64_t h = m.h, s = m.s, V = m.V, f = m.f, bw = m.bw, bo = m.bo;
  const int64_t b = pr.b, TP = pr.tp, DP = pr.dp;
  const int64_t first = (k == PP) ? 1 : 0;
  const int64_t last = (k == 1) ? 1 : 0;
  const int64_t dh = h / m.heads;
  const int64_t hkvr = (TP <= m.kv) ? (m.kv * dh) / TP : dh;  // KV heads replicated past kv
  const int64_t Pq = 2 * h * h;
  const int64_t Pm = (m.gpt ? 2 : 3) * h * f;
  const int64_t Prep = m.gpt ? 4 * h : 2 * h;
  const int64_t Psi = (Pq + Pm) / TP + 2 * h * hkvr + Prep;
  const int64_t Vr = (V + TP - 1) / TP;
  const int64_t Pe = Vr * h + (m.gpt ? s * h : 0);
  const int64_t Ph = Vr * h + (m.gpt ? 2 * h : h);
  const int64_t Pst = l * Psi + first * Pe + last * Ph;
  int64_t Pbuf = Psi;
  if (first * Pe > Pbuf) Pbuf = first * Pe;
  if (last * Ph > Pbuf) Pbuf = last * Ph;
  const int64_t mf = m.gpt ? 2 : 3;
  const int64_t atok = 4 * h + (2 * h + mf * f) / TP + 2 * hkvr + (m.flash ? 0 : m.heads * s / TP);
  const int64_t ftok = 2 * ((Pq + Pm) / TP + 2 * h * hkvr) + 4 * s * h / TP;
  const int64_t Fl = b * s * ftok;
  const int64_t Fh = last * 2 * b * s * h * Vr;
  const int64_t Xl = last * 4 * b * s * Vr;
  const int64_t p2pB = ((k > 1 ? 1 : 0) + (k < PP ? 1 : 0)) * b * s * h * bw;
  const int64_t arB = 2 * (TP - 1) * (b * s * h * bw / TP);
  const int64_t rB = (DP - 1) * bw * Pst;

  PairK P;
  P.afull = b * s * bw * atok;
  P.ack = b * s * bw * h;
  P.iD = pr.inv_dp;
  P.Pw = (double)(Pst * bw);
  P.Po = (double)(Pst * bo);
  P.Wb2 = (double)(2 * Pbuf * bw);
  P.Ob2o = (double)(2 * Pbuf * bo);
  P.A2 = (double)(2 * P.afull);
  P.AF = (double)P.afull;
  P.Xd = (double)Xl;
  P.Fld = (double)Fl;
  P.Fh3 = (double)(3 * Fh);
  P.r = ((double)rB * P.iD) * hw.iL;
  P.p2p = (double)p2pB * hw.iL;
  P.ar = (double)arB * hw.iL;
  P.FE = hw.iF * hw.ieta[pr.mb];
  return P;
}

struct CkptK {
  double A, KA, Rc, C;  // microbatch activations, in-flight stash, recompute unit, compute time
};

__device__ __forceinline__ CkptK ckpt_level(const PairK& P, int64_t l, int64_t c, int64_t ke) {
  const int64_t Amb = (l - c) * P.afull + c * P.ack;
  CkptK K;
  K.A = (double)Amb;
  K.KA = (double)(ke * Amb);
  K.Rc = c > 0 ? P.AF : 0.0;
  // fwd + 2 bwd per layer, one more fwd per recomputed layer, LM head fwd + bwd; serial TP
  // all-reduces: 2 fwd + 2 bwd per layer, 2 per recomputed layer.
  const double work = __builtin_fma((double)(3 * l + c), P.Fld, P.Fh3);
  K.C = __builtin_fma((double)(4 * l + 2 * c), P.ar, work * P.FE);
  return K;
}

struct ZeroK {
  double sw, sg;       // shard factors of weights and gradients
  double Sw, Sg, So;   // resident-if-kept bytes: weights, gradients, optimizer states
  double HWz;          // weight bytes fetched per microbatch (forward and backward)
  double G2Gs, G2Gf;   // GPU<->GPU stream: stable and first microbatch
  double Obo, Obg;     // optimizer-step unit parts
};

__device__ __forceinline__ ZeroK zero_level(const PairK& P, int z) {
  ZeroK Z;
  Z.sw = z == 3 ? P.iD : 1.0;
  Z.sg = z >= 2 ? P.iD : 1.0;
  const double so = z >= 1 ? P.iD : 1.0;
  Z.Sw = P.Pw * Z.sw;
  Z.Sg = P.Pw * Z.sg;
  Z.So = P.Po * so;
  Z.HWz = 2.0 * Z.Sw;
  const double ms = z == 2 ? 1.0 : (z == 3 ? 3.0 : 0.0);  // RS; AG + AG + RS
  const double mf = z == 3 ? 3.0 : 2.0;                   // first microbatch in total
  Z.G2Gs = __builtin_fma(ms, P.r, P.p2p);
  Z.G2Gf = __builtin_fma(mf, P.r, P.p2p);
  Z.Obo = P.Ob2o * so;
  Z.Obg = P.Wb2 * Z.sg;
  return Z;
}

// Everything of one configuration that does not depend on the activation offload ratio.
struct OuterK {
  double Bmax;         // max(forward, backward) peak without the activation terms
  double HW, DG;       // bytes: weights in, gradients out per microbatch
  double H2Dx, D2Hx;   // seconds: first-microbatch extras
};

__device__ __forceinline__ OuterK offload_levels(const PairK& P, const CkptK& K, const ZeroK& Z,
                                                 double rw, double qw, double rg, double qg,
                                                 double ro, double qo, double iP) {
  // weight offload
  const double Sww = qw * Z.Sw;
  const double Wbuf = P.Wb2 * (1.0 - qw * Z.sw);
  const double HW = rw * Z.HWz;
  const double DW = rw * Z.Sw;
  // gradient offload
  const double Swg = __builtin_fma(qg, Z.Sg, Sww);
  const double Gbuf = P.Wb2 * (1.0 - qg * Z.sg);
  const double DG = rg * Z.Sg;
  const double Og = rg * Z.Obg;
  // optimizer-state offload
  const double S = __builtin_fma(qo, Z.So, Swg);
  const double Obuf = __builtin_fma(ro, Z.Obo, Og);
  const double HX = __builtin_fma(ro, Z.So, DG);
  const double DX = __builtin_fma(ro, Z.So, DW);
  const double base = S + Wbuf;
  const double BF = (base + Obuf) + P.Xd;
  const double BB = ((base + Gbuf) + K.Rc) + P.Xd;
  OuterK O;
  // max(BF + x, BB + x) == max(BF, BB) + x: rounding to nearest is monotone.
  O.Bmax = __builtin_fmax(BF, BB);
  O.HW = HW;
  O.DG = DG;
  O.H2Dx = HX * iP;
  O.D2Hx = DX * iP;
  return O;
}

// Algorithm 1.  Repeatedly, while at least two streams still run, the streams of the
// current co-running pattern are scaled by that pattern's slowdown factors, the smallest
// scaled time overlaps all of them, and the others keep their remaining standalone time;
// the leftover stream's time is added at the end.  Visiting n = 4..2 and updating when the
// pattern has exactly n streams is the same as updating while the pattern has >= 2 streams,
// since every update stops at least one stream.  Absent streams carry factor +inf: their
// zero time scales to NaN, which the minimum skips and the final max(., 0) turns back to 0.
__device__ __forceinline__ double interference(double x0, double x1, double x2, double x3,
                                               const double* __restrict__ tab) {
  double T = 0.0;
#pragma unroll
  for (int it = 0; it < 3; ++it) {
    const int pat = (x0 != 0.0 ? 1 : 0) | (x1 != 0.0 ? 2 : 0) | (x2 != 0.0 ? 4 : 0) |
                    (x3 != 0.0 ? 8 : 0);
    if (__popc(pat) < 2) break;
    const double* e = tab + pat * kTabStride;
    const double s0 = x0 * e[0], s1 = x1 * e[1], s2 = x2 * e[2], s3 = x3 * e[3];
    const double ov = __builtin_fmin(__builtin_fmin(s0, s1), __builtin_fmin(s2, s3));
    x0 = __builtin_fmax((s0 - ov) * e[4], 0.0);
    x1 = __builtin_fmax((s1 - ov) * e[5], 0.0);
    x2 = __builtin_fmax((s2 - ov) * e[6], 0.0);
    x3 = __builtin_fmax((s3 - ov) * e[7], 0.0);
    T = T + ov;
  }
  T = T + x0;
  T = T + x1;
  T = T + x2;
  T = T + x3;
  return T;
}

struct Result {
  double t, d, mem, obj;
};

__device__ __forceinline__ Result config_level(const CkptK& K, const ZeroK& Z, const OuterK& O,
                                               double ra, double qa, double A2, double iP,
                                               double Gd, const double* tab) {
  Result r;
  const double SO = __builtin_fma(ra, A2, qa * K.KA);  // stash + double-buffered offload
  r.mem = O.Bmax + SO;
  const double H2Ds = __builtin_fma(ra, K.A, O.HW) * iP;
  const double D2Hs = __builtin_fma(ra, K.A, O.DG) * iP;
  const double H2Df = H2Ds + O.H2Dx;
  const double D2Hf = D2Hs + O.D2Hx;
  r.t = interference(K.C, Z.G2Gs, H2Ds, D2Hs, tab);
  const double T1 = interference(K.C, Z.G2Gf, H2Df, D2Hf, tab);
  r.d = T1 - r.t;
  r.obj = __builtin_fma(Gd, r.t, r.d);
  return r;
}

// Bucket j = min{j : mem <= edge[j]} for a feasible mem (mem <= edge[NB-1]).  The estimate
// floor(mem * NB / M) is within one of j; the loops settle it against the edges.
__device__ __forceinline__ int bucket_of(double mem, double kNB, const double* edge, int NB) {
  int j = (int)(mem * kNB);
  j = j < NB - 1 ? j : NB - 1;
  while (j < NB - 1 && mem > edge[j]) ++j;
  while (j > 0 && mem <= edge[j - 1]) --j;
  return j;
}

// ---------------------------------------------------------------------------------------
// K1: one block per tile (units of one group).  Wave w takes units w, w+4, ...; a unit is
// one (pair, c) slab; its lanes take the (z, wo, go, oo) slots; each lane walks the R
// activation ratios.  Every wave keeps a private LDS table of the 64 bucket minima; the
// block merges them into the tile's partials.
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_eval(EvalArgs a) {
  __shared__ double s_tab[16 * kTabStride];
  __shared__ double s_edge[MIST_MAX_BUCKETS];
  __shared__ double s_r[MIST_MAX_RATIOS];
  __shared__ double s_om[MIST_MAX_RATIOS];
  __shared__ double w_obj[kWaves][64];
  __shared__ uint64_t w_id[kWaves][64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const DevTile tile = a.tiles[blockIdx.x];
  const DevGroup g = a.groups[tile.group];
  const DevHw& hw = a.hws[g.hw];
  const int R = a.R, NB = a.NB, F = a.F;

  for (int i = tid; i < 16 * kTabStride; i += kBlock) s_tab[i] = (&hw.itab[0][0])[i];
  if (tid < MIST_MAX_BUCKETS) s_edge[tid] = hw.edge[tid];
  if (tid < R) {
    s_r[tid] = a.ratio[tid];
    s_om[tid] = a.ratio[R + tid];
  }
  w_obj[wave][lane] = __builtin_huge_val();
  w_id[wave][lane] = kNone;
  __syncthreads();

  const double iP = hw.iP, M = hw.M, kNB = hw.kNB;
  const int64_t l = g.l;
  const int64_t ke = g.k < g.G ? g.k : g.G;
  const double Gd = (double)g.G;

  for (int u = tile.unit_begin + wave; u < tile.unit_end; u += kWaves) {
    const int p = u / (g.l + 1);
    const int c = u - p * (g.l + 1);
    const DevPair pr = a.pairs[g.pair_begin + p];
    const PairK P = pair_level(a.m, g.PP, g.k, l, pr, hw);
    const CkptK K = ckpt_level(P, l, c, ke);
    const uint64_t unit_id = g.base + (uint64_t)u * (uint64_t)F * (uint64_t)R;

    for (int f = lane; f < F; f += 64) {
      int v = f;
      const int io = v % R;
      v /= R;
      const int ig = v % R;
      v /= R;
      const int iw = v % R;
      const int z = v / R;
      const ZeroK Z = zero_level(P, z);
      const OuterK O = offload_levels(P, K, Z, s_r[iw], s_om[iw], s_r[ig], s_om[ig], s_r[io],
                                      s_om[io], iP);
      const uint64_t id0 = unit_id + (uint64_t)f * (uint64_t)R;

      for (int ia = 0; ia < R; ++ia) {
        const Result r = config_level(K, Z, O, s_r[ia], s_om[ia], P.A2, iP, Gd, s_tab);
        const uint64_t id = id0 + (uint64_t)ia;
        const bool feasible = r.mem <= M;
        const int j = feasible ? bucket_of(r.mem, kNB, s_edge, NB) : 0;
        bool cand = feasible && lex_less(r.obj, id, w_obj[wave][j], w_id[wave][j]);
        uint64_t ballot = __ballot(cand);
        while (ballot) {
          const int leader = __ffsll((unsigned long long)ballot) - 1;
          if (lane == leader) {
            if (lex_less(r.obj, id, w_obj[wave][j], w_id[wave][j])) {
              w_obj[wave][j] = r.obj;
              w_id[wave][j] = id;
            }
            cand = false;
          }
          __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
          __builtin_amdgcn_wave_barrier();
          if (cand) cand = lex_less(r.obj, id, w_obj[wave][j], w_id[wave][j]);
          ballot = __ballot(cand);
        }
      }
    }
  }
  __syncthreads();
  if (tid < 64) {
    double bo = w_obj[0][tid];
    uint64_t bi = w_id[0][tid];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
      if (lex_less(w_obj[w][tid], w_id[w][tid], bo, bi)) {
        bo = w_obj[w][tid];
        bi = w_id[w][tid];
      }
    }
    a.part_obj[(size_t)blockIdx.x * 64 + tid] = bo;
    a.part_id[(size_t)blockIdx.x * 64 + tid] = bi;
  }
}

// ---------------------------------------------------------------------------------------
// K2: one wave per group; lane j owns bucket j.  Lexicographic minimum over the group's
// tiles in tile order, then the group's best by a butterfly over the 64 lanes and the
// staircase by an exclusive prefix minimum over the buckets.
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kReduceBlock) void k_reduce(ReduceArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * (kReduceBlock / 64) + (threadIdx.x >> 6);
  if (g >= a.n_groups) return;
  const DevGroup grp = a.groups[g];
  double obj = __builtin_huge_val();
  uint64_t id = kNone;
  if (lane < a.NB) {
    for (int t = grp.tile_begin; t < grp.tile_begin + grp.n_tiles; ++t) {
      const double o = a.part_obj[(size_t)t * 64 + lane];
      const uint64_t i = a.part_id[(size_t)t * 64 + lane];
      if (lex_less(o, i, obj, id)) {
        obj = o;
        id = i;
      }
    }
  }
  a.bucket_obj[g * 64 + lane] = obj;
  a.bucket_id[g * 64 + lane] = id;

  double bo = obj;
  uint64_t bi = id;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const double o = __shfl_xor(bo, off, 64);
    const uint64_t i = __shfl_xor(bi, off, 64);
    if (lex_less(o, i, bo, bi)) {
      bo = o;
      bi = i;
    }
  }
  double pm = obj;  // inclusive prefix minimum over buckets 0..lane
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(pm, off, 64);
    if (lane >= off) pm = __builtin_fmin(pm, o);
  }
  double below = __shfl_up(pm, 1, 64);
  if (lane == 0) below = __builtin_huge_val();
  const bool on = id != kNone && obj < below;
  const uint64_t mask = __ballot(on);
  if (lane == 0) {
    a.best_obj[g] = bo;
    a.best_id[g] = bi;
    a.frontier[g] = mask;
  }
}

// ---------------------------------------------------------------------------------------
// Per-id evaluation with the same level functions (parity and result extraction).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_eval_ids(EvalArgs a, const uint64_t* __restrict__ ids,
                                                  int64_t n, double* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t id = ids[i];
  int64_t lo = 0, hi = a.n_groups;
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) / 2;
    if (a.groups[mid].base <= id) lo = mid;
    else hi = mid;
  }
  const DevGroup g = a.groups[lo];
  const DevHw& hw = a.hws[g.hw];
  const uint64_t R = (uint64_t)a.R;
  uint64_t v = id - g.base;
  const int ia = (int)(v % R);
  v /= R;
  const int io = (int)(v % R);
  v /= R;
  const int ig = (int)(v % R);
  v /= R;
  const int iw = (int)(v % R);
  v /= R;
  const int z = (int)(v % 4);
  v /= 4;
  const int c = (int)(v % (uint64_t)(g.l + 1));
  const int p = (int)(v / (uint64_t)(g.l + 1));
  const double* r = a.ratio;
  const double* om = a.ratio + a.R;
  const int64_t ke = g.k < g.G ? g.k : g.G;
  const PairK P = pair_level(a.m, g.PP, g.k, g.l, a.pairs[g.pair_begin + p], hw);
  const CkptK K = ckpt_level(P, g.l, c, ke);
  const ZeroK Z = zero_level(P, z);
  const OuterK O = offload_levels(P, K, Z, r[iw], om[iw], r[ig], om[ig], r[io], om[io], hw.iP);
  const Result res = config_level(K, Z, O, r[ia], om[ia], P.A2, hw.iP, (double)g.G, &hw.itab[0][0]);
  out[4 * i + 0] = res.t;
  out[4 * i + 1] = res.d;
  out[4 * i + 2] = res.mem;
  out[4 * i + 3] = res.obj;
}

int check_launch() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace

int launch_eval(const EvalArgs& a, void* stream) {
  if (a.n_tiles <= 0) return 0;
  hipLaunchKernelGGL(k_eval, dim3(a.n_tiles), dim3(kBlock), 0, (hipStream_t)stream, a);
  return check_launch();
}

int launch_reduce(const ReduceArgs& a, void* stream) {
  if (a.n_groups <= 0) return 0;
  const int per = kReduceBlock / 64;
  const int64_t blocks = (a.n_groups + per - 1) / per;
  hipLaunchKernelGGL(k_reduce, dim3((unsigned)blocks), dim3(kReduceBlock), 0, (hipStream_t)stream, a);
  return check_launch();
}

int launch_eval_ids(const EvalArgs& a, const uint64_t* ids, int64_t n, double* out, void* stream) {
  if (n <= 0) return 0;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(k_eval_ids, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, a, ids,
                     n, out);
  return check_launch();
}

}  // namespace mist
