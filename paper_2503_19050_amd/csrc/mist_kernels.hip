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

// Weight and gradient offload levels (fixed within a strip).
struct WoGoK {
  double Swg;          // resident weight + gradient bytes
  double Wbuf, Gbuf;   // double-buffered fetched weights / gradient unit
  double HW;           // weight bytes fetched per microbatch (forward and backward)
  double DW;           // updated weight bytes written back after the step
  double DG;           // gradient bytes offloaded per microbatch
  double Og;           // gradient part of the optimizer-step unit
};

__device__ __forceinline__ WoGoK wogo_levels(const PairK& P, const ZeroK& Z, double rw, double qw,
                                             double rg, double qg) {
  WoGoK W;
  const double Sww = qw * Z.Sw;
  W.Wbuf = P.Wb2 * (1.0 - qw * Z.sw);
  W.HW = rw * Z.HWz;
  W.DW = rw * Z.Sw;
  W.Swg = __builtin_fma(qg, Z.Sg, Sww);
  W.Gbuf = P.Wb2 * (1.0 - qg * Z.sg);
  W.DG = rg * Z.Sg;
  W.Og = rg * Z.Obg;
  return W;
}

// Strip constants that the optimizer-state offload level reads, kept in a per-lane LDS
// record (registers are the scarce resource of the evaluation kernel).
struct OoIn {
  double So, Swg, Obo, Og, DG, DW, Wbuf, Gbuf, Rc, Xd;
};

// Optimizer-state offload level: everything of a configuration except its activation
// ratio's terms.
struct OoK {
  double Bmax;         // max(forward, backward) peak without the activation terms
  double H2Dx, D2Hx;   // seconds: first-microbatch extras
};

__device__ __forceinline__ OoIn oo_inputs(const PairK& P, const CkptK& K, const ZeroK& Z,
                                          const WoGoK& W) {
  return OoIn{Z.So, W.Swg, Z.Obo, W.Og, W.DG, W.DW, W.Wbuf, W.Gbuf, K.Rc, P.Xd};
}

__device__ __forceinline__ OoK oo_level(const OoIn& I, double ro, double qo, double iP) {
  const double S = __builtin_fma(qo, I.So, I.Swg);
  const double Obuf = __builtin_fma(ro, I.Obo, I.Og);
  const double HX = __builtin_fma(ro, I.So, I.DG);
  const double DX = __builtin_fma(ro, I.So, I.DW);
  const double base = S + I.Wbuf;
  const double BF = (base + Obuf) + I.Xd;
  const double BB = ((base + I.Gbuf) + I.Rc) + I.Xd;
  OoK O;
  // max(BF + x, BB + x) == max(BF, BB) + x: rounding to nearest is monotone.
  O.Bmax = __builtin_fmax(BF, BB);
  O.H2Dx = HX * iP;
  O.D2Hx = DX * iP;
  return O;
}

// ---------------------------------------------------------------------------------------
// Algorithm 1.
//
// Visiting n = 4..2 and updating when the non-zero pattern has exactly n streams is the
// same as updating while the pattern has at least two streams (each update stops at least
// one stream), so three fixed rounds suffice.  A round reads the row of the current
// pattern: rows of two or more streams scale members by phi, overlap the smallest scaled
// time, and leave members (scaled - overlap) * psi; non-members (time 0, or NaN from an
// earlier round) carry phi = +inf and become NaN, which min and max skip and "> 0"
// rejects.  Rows of at most one stream have phi = psi = 1; such a round always meets an
// exact zero (an unused stream, or the stream that finished last) so its overlap is 0 and
// nothing changes.  At the end at most one stream is positive and the others are 0 or NaN,
// so the oracle's final sum equals the running total plus the largest remaining time.
// ---------------------------------------------------------------------------------------
struct Streams {
  double x0, x1, x2, x3;
};

__device__ __forceinline__ double round_row(Streams& x, double f0, double f1, double f2, double f3,
                                            double p0, double p1, double p2, double p3) {
  const double s0 = x.x0 * f0, s1 = x.x1 * f1, s2 = x.x2 * f2, s3 = x.x3 * f3;
  const double ov = __builtin_fmin(__builtin_fmin(s0, s1), __builtin_fmin(s2, s3));
  x.x0 = (s0 - ov) * p0;
  x.x1 = (s1 - ov) * p1;
  x.x2 = (s2 - ov) * p2;
  x.x3 = (s3 - ov) * p3;
  return ov;
}

// Interference rows in LDS are padded to kLdsRow doubles so that lanes reading different
// rows spread over more banks.
constexpr int kLdsRow = 10;

template <int STRIDE>
__device__ __forceinline__ double round_lookup(Streams& x, const double* __restrict__ tab) {
  // Row of the non-zero pattern (bit i for stream i), as a pre-scaled offset.
  const int off = (x.x0 > 0.0 ? STRIDE : 0) + (x.x1 > 0.0 ? 2 * STRIDE : 0) +
                  (x.x2 > 0.0 ? 4 * STRIDE : 0) + (x.x3 > 0.0 ? 8 * STRIDE : 0);
  const double* e = tab + off;
  return round_row(x, e[0], e[1], e[2], e[3], e[4], e[5], e[6], e[7]);
}

__device__ __forceinline__ double remaining(const Streams& x) {
  return __builtin_fmax(__builtin_fmax(x.x0, x.x1), __builtin_fmax(x.x2, x.x3));
}

// Three rounds with per-lane rows (rows STRIDE doubles apart).
template <int STRIDE = kLdsRow>
__device__ __forceinline__ double interference(double c, double g, double h, double d,
                                               const double* __restrict__ tab) {
  Streams x{c, g, h, d};
  double T = round_lookup<STRIDE>(x, tab);
  T = T + round_lookup<STRIDE>(x, tab);
  T = T + round_lookup<STRIDE>(x, tab);
  return T + remaining(x);
}

// Calls whose first round uses a row known in advance: every configuration of a strip whose host
// streams both run (pattern 15, or 13 without GPU-GPU traffic), with compute c and GPU-GPU g fixed
// per strip.  The strip precomputes the scaled c and g and their minimum m01.
//
// After a round a member keeps running exactly when its scaled time exceeds the overlap
// (s_j - ov > 0, and (s_j - ov) * psi_j cannot round to zero: the host's input bounds keep every
// non-zero stream time and difference far above the subnormal range).  In the common case the
// GPU-GPU stream is a member and its scaled time s1 is below every other member's: the overlap is
// s1 itself, compute, host->device and device->host keep running, and the second round reads
// row 13 for every such configuration, with compute's second-round scaled time y0 fixed per
// strip.  The second-round scaled times y_j = ((s_j - s1) * psi15_j) * phi13_j have the sign of
// s_j - s1, so that case is y0 > 0 and y2, y3 > 0 (with pattern 13, s1 and y0 are NaN and the
// case never holds).
struct KnownRow {
  double s0, s1, m01;   // c * phi0, g * phi1 (NaN when GPU-GPU is no member), min of the two
  double y0;            // compute's scaled time in the second round (row 13) when s1 < s0
  const double* row;    // the first round's row
};

__device__ __forceinline__ KnownRow known_row(const double* __restrict__ tab, int pattern, double c, double g) {
  const double* e = tab + pattern * kLdsRow;
  KnownRow r;
  r.s0 = c * e[0];
  r.s1 = g * e[1];
  r.m01 = __builtin_fmin(r.s0, r.s1);
  r.row = e;
  r.y0 = ((r.s0 - r.s1) * e[4]) * tab[13 * kLdsRow + 0];
  return r;
}

// General rounds of such a call with host streams h, d > 0: the first with the known row, the
// others looked up by the lanes' patterns.
__device__ __forceinline__ double interference_general(const KnownRow& r, double h, double d,
                                                       const double* __restrict__ tab) {
  const double* e = r.row;
  const double s2 = h * e[2], s3 = d * e[3];
  const double ov = __builtin_fmin(r.m01, __builtin_fmin(s2, s3));
  Streams x{(r.s0 - ov) * e[4], (r.s1 - ov) * e[5], (s2 - ov) * e[6], (s3 - ov) * e[7]};
  double T = ov;
  T = T + round_lookup<kLdsRow>(x, tab);
  T = T + round_lookup<kLdsRow>(x, tab);
  return T + remaining(x);
}

// Rows of the third round when compute and one host stream are left after the second round
// (row 13's overlap ended the other host stream): for the stream h left (index 0: h = 2, row 5;
// index 1: h = 3, row 9) the kTab2 doubles phi[0], phi[h], psi[0], psi[h] of that row and psi[0],
// psi[h] of row 13, so that a lane reads its row from one per-lane offset.
constexpr int kTab2 = 6;
constexpr int kTab2Off = 16 * kLdsRow;  // after the sixteen pattern rows

// The factors every configuration's second-round scaled host times read: phi and psi of the host
// streams in row 15 and their phi in row 13.  Wave-uniform, loaded once per tile into scalar
// registers (as vector registers they crowd the strip loop into spilling).
struct RowK {
  double f2, f3;  // phi15[2], phi15[3]
  double p2, p3;  // psi15[2], psi15[3]
  double g2, g3;  // phi13[2], phi13[3]
};

// Algorithm 1 for one configuration of a strip with the strip's known first-round row.  Each form
// is chosen for the whole wave (lanes with free set, whose result the caller replaces or does
// not use, do not take part), so that every form is straight-line code:
//   - GPU-GPU finishes first (row 15) and the second round (row 13: compute, host->device,
//     device->host) ends the smaller host stream: compute and the larger host stream are left,
//     and each lane reads their row (5 or 9) at a per-lane offset and forms only their terms;
//   - GPU-GPU finishes first and compute ends the second round: both host streams are left, and
//     the third round's row (12) is the same for the wave;
//   - GPU-GPU finishes first otherwise (waves that mix the two cases above, ties): the third
//     round's row is looked up per lane from all three streams;
//   - else the general rounds (interference_general).
// Each form performs the same operations on the same operands as the general rounds: a stream
// that has finished carries NaN there (its time 0 times the row's +inf factor), which drops out
// of the minimum and the maximum that the special forms take over the streams left.  form
// receives the form taken (kForm*; read by the dump variant only).
constexpr int kFormHostLeft = 1;    // compute and the larger host stream left: per-lane row 5 or 9
constexpr int kFormHostsLeft = 2;   // compute finished in the second round: row 12
constexpr int kFormLookup = 3;      // GPU-GPU first, third row looked up per lane
constexpr int kFormGeneral = 4;     // the general rounds
constexpr int kFormZero = 5;        // the all-zero configuration's closed form (first microbatch)
constexpr int kFormGeneric = 6;     // three rounds from an unknown pattern (stable time, ratio 0)

__device__ __forceinline__ double interference_known(const KnownRow& r, double h, double d, bool free,
                                                     const double* __restrict__ tab, const RowK& K,
                                                     int& form) {
  const double* e13 = tab + 13 * kLdsRow;
  const double y0 = r.y0;
  const double y2 = ((h * K.f2 - r.s1) * K.p2) * K.g2;
  const double y3 = ((d * K.f3 - r.s1) * K.p3) * K.g3;
  const double m23 = __builtin_fmin(y2, y3);
  const double yh = __builtin_fmax(y2, y3);
  // Wave masks of plain compares (combined by the scalar unit).
  const unsigned long long ex = __builtin_amdgcn_read_exec();
  const unsigned long long fm = __builtin_amdgcn_ballot_w64(free);
  const unsigned long long g1 = __builtin_amdgcn_ballot_w64(m23 > 0.0);  // with y0 > 0: GPU-GPU first
  if (((__builtin_amdgcn_ballot_w64(y0 > m23) & g1 & __builtin_amdgcn_ballot_w64(yh > m23)) | fm) == ex) {
    // Compute and the larger host stream are left (row 5 or 9); the second round's overlap is
    // the smaller host time m23.
    const double* e = tab + kTab2Off + (y2 > y3 ? 0 : kTab2);
    const double z0 = (y0 - m23) * e[4];
    const double zh = (yh - m23) * e[5];
    const double w0 = z0 * e[0], wh = zh * e[1];
    const double ov3 = __builtin_fmin(w0, wh);
    const double rem = __builtin_fmax((w0 - ov3) * e[2], (wh - ov3) * e[3]);
    form = kFormHostLeft;
    return ((r.s1 + m23) + ov3) + rem;
  }
  const unsigned long long y0p = __builtin_amdgcn_ballot_w64(y0 > 0.0);
  if (((__builtin_amdgcn_ballot_w64(y0 < m23) & y0p) | fm) == ex) {
    // Compute finished in the second round (overlap y0); both host streams are left (row 12).
    const double* e12 = tab + 12 * kLdsRow;
    const double w2 = ((y2 - y0) * e13[6]) * e12[2];
    const double w3 = ((y3 - y0) * e13[7]) * e12[3];
    const double ov3 = __builtin_fmin(w2, w3);
    const double rem = __builtin_fmax((w2 - ov3) * e12[6], (w3 - ov3) * e12[7]);
    form = kFormHostsLeft;
    return ((r.s1 + y0) + ov3) + rem;
  }
  if (((y0p & g1) | fm) == ex) {
    const double ov2 = __builtin_fmin(y0, m23);
    const double T2 = r.s1 + ov2;
    // Third round: the row of the streams still running, those whose scaled time exceeds the
    // overlap.
    const bool q0 = y0 > ov2, q2 = y2 > ov2, q3 = y3 > ov2;
    const double z0 = (y0 - ov2) * e13[4], z2 = (y2 - ov2) * e13[6], z3 = (y3 - ov2) * e13[7];
    const double* e = tab + ((q0 ? 1 : 0) + (q2 ? 4 : 0) + (q3 ? 8 : 0)) * kLdsRow;
    const double w0 = z0 * e[0], w2 = z2 * e[2], w3 = z3 * e[3];
    const double ov3 = __builtin_fmin(__builtin_fmin(w0, w2), w3);
    const double rem = __builtin_fmax(__builtin_fmax((w0 - ov3) * e[4], (w2 - ov3) * e[6]), (w3 - ov3) * e[7]);
    form = kFormLookup;
    return (T2 + ov3) + rem;
  }
  form = kFormGeneral;
  return interference_general(r, h, d, tab);
}

// Algorithm 1 for the first n of the N configurations of an activation-ratio block (host streams
// h[c], d[c]), one wave-uniform choice of form per configuration (measured fastest against one
// choice per block or half block: 0.81 against 1.16 and 1.02 ms on gpt2.7b-d16, equal on the
// Llama spaces).  With SKIP a configuration free in every lane is not evaluated, and every free
// lane's result is NaN.
template <int N, bool SKIP = false>
__device__ __forceinline__ void interference_known_n(const KnownRow& r, const double (&h)[N], const double (&d)[N],
                                                     const bool (&free)[N], double (&out)[N], int (&form)[N], int n,
                                                     const double* __restrict__ tab, const RowK& K) {
#pragma unroll
  for (int c = 0; c < N; ++c) {
    if (c >= n) break;
    form[c] = 0;
    if (SKIP && !__builtin_amdgcn_ballot_w64(!free[c]))  // every lane's result is unused: none is formed
      out[c] = __builtin_nan("");
    else
      out[c] = interference_known(r, h[c], d[c], free[c], tab, K, form[c]);
    if constexpr (SKIP) out[c] = free[c] ? __builtin_nan("") : out[c];
  }
}

// Algorithm 1 on (c, g, +0, +0), c > 0: the first round uses the row of pattern 3 (compute and
// GPU-GPU), after which at most one stream is positive and the other rounds leave the times
// unchanged and add +0; with g = 0 the only row met has one stream and the time is c.  This
// equals interference() on the same streams bit for bit.
__device__ __forceinline__ double interference_zero(double c, double g, const double* __restrict__ tab) {
  const double* e = tab + 3 * kLdsRow;
  const double s0 = c * e[0], s1 = g * e[1];
  const double ov = __builtin_fmin(s0, s1);
  const double t = ov + __builtin_fmax((s0 - ov) * e[4], (s1 - ov) * e[5]);
  return g > 0.0 ? t : c;
}

// K0: pair-level constants of every (group, pair).
__global__ __launch_bounds__(256) void k_pairs(EvalArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < kClaimCounters) a.work[i * kCounterStride] = 0;  // the evaluation kernel's tile
                                                           // counters (it runs after this one)
  if (i == 0 && a.pool_count) *a.pool_count = 0ull;       // and its candidate overflow pool
  if (i >= a.n_pk) return;
  const DevGroup g = a.groups[a.pk_group[i]];
  const int p = i - g.pk_begin;
  a.pk[i] = pair_level(a.m, g.PP, g.k, g.l, a.pairs[g.pair_begin + p], a.hws[g.hw]);
}

// ---------------------------------------------------------------------------------------
// K1.  Persistent: every wave takes one tile (a range of strips of one group) by its index
// in the grid and claims further tiles from a device counter until none is left; each lane
// walks the tile's strips with stride 64.  A
// strip fixes (pair, c, z, wo, go) and holds the R x R (optimizer ratio, activation ratio)
// configurations:
//   - the stable time t does not depend on the optimizer ratio, so it is computed once per
//     activation ratio and reused across the optimizer ratios;
//   - the first microbatch's streams start in the same pattern for every configuration of
//     the strip (compute, GPU-GPU iff that stream carries traffic, and both host streams
//     iff any offload ratio is non-zero), except the one configuration whose four ratios
//     are all zero: its host streams are exactly +0, and its time is computed once per
//     strip in closed form (interference_zero).
// Each wave keeps an LDS table of the 64 bucket minima of its current tile and writes it
// as the tile's partials.
// ---------------------------------------------------------------------------------------
struct BucketEntry {
  double edge;             // the bucket's upper memory edge E_j (+inf past NB - 1): the edge
                           // and the key are adjacent, read together
  unsigned long long key;  // bits of the minimum objective (a non-negative double orders like
                           // its bit pattern)
  unsigned int lid;        // lowest local id (id - group base, < 2^32) reaching it
  unsigned int pad;
};
static_assert(sizeof(BucketEntry) == 24, "24-byte entries: the entry offset is one multiply-add");

// Weight-sampled argmin (Eq. 4 with sampled alpha) of the wave's current tile: the value
// (a double, for the fast comparison), its order key (for the LDS atomic minimum; weighted
// values may be negative) and the lowest local id reaching it.
struct AlphaEntry {
  double val;
  unsigned long long key;
  unsigned int lid;
  unsigned int pad;
};

// Reads a table entry at a wave-uniform index through the constant address space, so that it
// arrives in scalar registers (scalar loads; the tables are read-only during the kernel).
template <class T>
__device__ __forceinline__ T load_uniform(const T* p) {
  static_assert(sizeof(T) % 4 == 0, "whole dwords");
  const __attribute__((address_space(4))) uint32_t* q = (const __attribute__((address_space(4))) uint32_t*)p;
  T v;
  uint32_t* d = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) d[i] = q[i];
  return v;
}

// A 64-bit key that orders like the double (neither -0 nor NaN occurs as a key).
__device__ __forceinline__ unsigned long long order_key(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

// Orders this wave's LDS accesses for the compiler: a lane may read a word another lane of
// the same wave wrote (the hardware executes a wave's LDS operations in order), so no load
// may be moved across this point or answered from the lane's own earlier store.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Words that other lanes of the wave update with atomics are read and written with relaxed
// wavefront-scope atomics: a plain load after a lane's own atomic update could otherwise be
// answered from a value the compiler already holds (for an entry at a wave-uniform address the
// compiler combines the lanes' atomic minima into one update by one lane).
template <class T>
__device__ __forceinline__ T lds_load(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

template <class T>
__device__ __forceinline__ void lds_store(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

// Overflow pool of the exact frontier's candidate pass: each wave takes chunks of kPoolChunk
// slots; the slots of a chunk it leaves unused are marked (tile -1) so that the placement skips
// them.
constexpr int kPoolChunk = 256;

__device__ __forceinline__ void pool_holes(const EvalArgs& a, unsigned long long base, int used, int lane) {
  // The active lanes share the work (lanes past a ragged tile's last strip are inactive).
  const unsigned long long ex = __builtin_amdgcn_read_exec();
  const int n_act = __builtin_popcountll(ex);
  const int r = (int)__builtin_amdgcn_mbcnt_hi((unsigned int)(ex >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)ex, 0u));
  (void)lane;
  for (int i = used + r; i < kPoolChunk; i += n_act) {
    const unsigned long long pos = base + (unsigned long long)i;
    if (pos < (unsigned long long)a.pool_cap) a.pool_tile[pos] = -1;
  }
}

// Activation ratios per block of the strip loop: a block keeps its stable times and the
// per-ratio terms of its configurations in registers across the optimizer ratios.
// Weight samples take larger blocks for 7 <= R <= 10 (at R = 9, 79.5 against 85.2 ms for 8
// samples on the 64-hardware-sample Llama space).
template <int R, int MODE>
constexpr int ia_block() {
  return R <= 6 ? R : (MODE == kModeAlpha && R <= 10 ? (R + 1) / 2 : (R + 2) / 3);
}

// A value every lane of the wave holds, moved to scalar registers.
__device__ __forceinline__ double wave_uniform(double x) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(x);
  const unsigned int lo = __builtin_amdgcn_readfirstlane((unsigned int)b);
  const unsigned int hi = __builtin_amdgcn_readfirstlane((unsigned int)(b >> 32));
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Waves per SIMD the register allocation aims at: four, 128 registers per lane (a few
// strip-level values spill; the occupancy is worth more).  Five would fit the LDS of the blocks,
// but at 96 registers the inner loop spills: 77 against 59 ms on the 64-sample Llama space.  The
// exact frontier's candidate variant keeps more per configuration live; with a whole strip's
// activation ratios in one block (R <= 6) three waves and fewer spills are faster (1.60 against
// 1.83 ms for the exact frontier on gpt2.7b-d16), with larger R four.
template <int R, int MODE>
constexpr int eval_waves() { return MODE == kModeEmit && R <= 6 ? 3 : 4; }

// MODE kModeBuckets: bucket minima; kModeAlpha: also the weight-sampled argmins of Eq. 4
// (a.n_alpha samples); kModeEmit: the exact frontier's candidates, written and counted per
// tile (the bucket reduction is skipped).
template <int R, int MODE>
__global__ __launch_bounds__(kBlock, (eval_waves<R, MODE>())) void k_eval(EvalArgs a, const double* __restrict__ ratio,
                                                                 const PairK* __restrict__ pk) {
  constexpr bool AL = MODE == kModeAlpha;
  constexpr bool EX = MODE == kModeEmit;
  constexpr bool DM = MODE == kModeDump;
  constexpr int R2 = R * R;
  constexpr int SU = 4 * R2;  // strips per (pair, c) unit
  constexpr int IB = ia_block<R, MODE>();
  // Exact frontier with the activation ratios in several blocks: lower bounds per strip and per
  // block (below).  With the whole strip in one block the candidates are dense and the bounds
  // rarely hold for a whole wave (1 % of the wave iterations on gpt2.7b-d16, simulated).
  constexpr bool BLK = EX && IB < R;
  __shared__ double s_tab[kWaves][16 * kLdsRow + 2 * kTab2];
  __shared__ BucketEntry s_bucket[kWaves][65];  // entries NB..64: sinks of infeasible configurations
  __shared__ OoIn s_oo[kBlock];         // per-lane strip constants of the optimizer level
  __shared__ double2 s_ab[AL ? kWaves : 1][kMaxAlphas];      // alpha * G, 1 - alpha
  __shared__ AlphaEntry s_aent[AL ? kWaves : 1][kMaxAlphas];
  __shared__ FiltEntry s_filt[EX ? kWaves : 1][EX ? 64 : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // The wave index is uniform across the wave: stated, so that the tile, group and hardware
  // values derived from it live in scalar registers (scalar loads) rather than in every lane.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int NB = a.NB;
  const double* __restrict__ rr = ratio;  // read-only and uniform: scalar loads
  const double* __restrict__ om = ratio + R;
  const bool r0_zero = rr[0] == 0.0;
  // The smallest offload ratio and the smallest 1 - r, for the strip bounds.
  [[maybe_unused]] double r_lo = 0.0, q_lo = 0.0;
  if constexpr (BLK) {
    r_lo = rr[0];
    q_lo = om[0];
    for (int i = 1; i < R; ++i) {
      r_lo = __builtin_fmin(r_lo, rr[i]);
      q_lo = __builtin_fmin(q_lo, om[i]);
    }
    r_lo = wave_uniform(r_lo);
    q_lo = wave_uniform(q_lo);
  }
  double* tab = s_tab[wave];
  BucketEntry* bucket = s_bucket[wave];
  const unsigned long long kEmpty = (unsigned long long)__double_as_longlong(__builtin_huge_val());

  // Tile schedule: wave w of the grid takes work item w.  Item n_waves + x + kClaimCounters
  // * c goes to the claim that draws number c from counter x (counters reset to 0 by K0); a
  // wave draws from the counter of its block's XCD and moves to the next counter when one
  // runs out, until all have.  When the grid has at least as many waves as there are items
  // no claim is made.  Item x is tile tile_order[x] (the host gives each XCD's items a
  // contiguous range of tiles), or tile tile_list[x] when a variant runs a list.
  const bool listed = (EX || DM) && a.tile_list != nullptr;
  const int n_items = listed ? a.n_list : a.n_tiles;
  const int n_waves = (int)gridDim.x * kWaves;
  const bool claims = n_items > n_waves;
  int counter = (int)(blockIdx.x % kClaimCounters);
  int exhausted = 0;
  int loaded_hw = -1;
  // Exact frontier: the wave's current chunk of overflow-pool slots (none yet: used = chunk).
  unsigned long long pool_base = 0;
  int pool_used = kPoolChunk;
  for (int x = (int)blockIdx.x * kWaves + wave; x < n_items;) {
    const int t = listed ? load_uniform(a.tile_list + x) : (a.tile_order ? load_uniform(a.tile_order + x) : x);
    const DevTile tile = load_uniform(a.tiles + t);
    // The exact frontier's pass skips a tile that holds no candidate (its count stays 0).
    const int strip_end = EX && a.tile_live && !a.tile_live[t] ? tile.strip_begin : tile.strip_end;
    const DevGroup g = load_uniform(a.groups + tile.group);
    const DevHw& hw = a.hws[g.hw];
    if (g.hw != loaded_hw) {  // the wave's LDS copy of the hardware tables
      for (int i = lane; i < 16 * kTabStride; i += 64)
        tab[(i / kTabStride) * kLdsRow + i % kTabStride] = (&hw.itab[0][0])[i];
      wave_sync();
      if (lane < 2 * kTab2) {  // the third round's rows of compute and one host stream, from the rows
        const int h = 2 + lane / kTab2, i = lane % kTab2;
        const int row = i < 4 ? (1 | (1 << h)) : 13;
        const int col = ((i & 1) ? h : 0) + (i >= 2 ? 4 : 0);  // phi[0], phi[h], psi[0], psi[h], psi[0], psi[h]
        tab[kTab2Off + lane] = tab[row * kLdsRow + col];
      }
      bucket[lane].edge = hw.edge[lane];
      loaded_hw = g.hw;
    }
    // Buckets 0..NB-1 start empty.  Entries NB..64 are sinks: they hold key 0 and local id
    // 0, which no configuration beats, so an infeasible configuration sent to one never
    // takes part.
    bucket[lane].key = lane < NB ? kEmpty : 0ull;
    bucket[lane].lid = lane < NB ? 0xFFFFFFFFu : 0u;
    if (lane == 0) {
      bucket[64].edge = __builtin_huge_val();
      bucket[64].key = 0ull;
      bucket[64].lid = 0u;
    }
    const double Gd = (double)g.G;
    int64_t n_cand = 0;  // exact frontier: the next candidate's slot
    int64_t n_beg = 0;   // and the tile's window of slots
    int64_t n_end = 0;
    bool dropped = false;  // and whether a candidate of this lane found no place
    if constexpr (EX) {
      s_filt[wave][lane] = a.filt[(size_t)tile.group * 64 + lane];
      n_beg = load_uniform(a.win_begin + t);  // wave-uniform: scalar registers
      n_end = load_uniform(a.win_end + t);
      n_cand = n_beg;
    }
    if constexpr (AL) {
      if (lane < a.n_alpha) {
        s_ab[wave][lane] = make_double2(a.alpha[lane] * Gd, a.beta[lane]);
        s_aent[wave][lane].val = __builtin_huge_val();
        s_aent[wave][lane].key = order_key(__builtin_huge_val());
        s_aent[wave][lane].lid = 0xFFFFFFFFu;
      }
    }
    wave_sync();

    const double iP = load_uniform(&hw.iP), kNB = load_uniform(&hw.kNB), M = load_uniform(&hw.M);
    const RowK RK{load_uniform(&hw.itab[15][2]), load_uniform(&hw.itab[15][3]), load_uniform(&hw.itab[15][6]),
                  load_uniform(&hw.itab[15][7]), load_uniform(&hw.itab[13][2]), load_uniform(&hw.itab[13][3])};
    const int l = g.l;
    const int64_t ke = g.k < g.G ? g.k : g.G;

#pragma unroll 1
    for (int s = tile.strip_begin + lane; s < strip_end; s += 64) {
      const int unit = s / SU;
      const int rem = s - unit * SU;
      const int z = rem / R2;
      const int rem2 = rem - z * R2;
      const int iw = rem2 / R;
      const int ig = rem2 - iw * R;
      const int p = unit / (l + 1);
      const int c = unit - p * (l + 1);
      const PairK P = pk[g.pk_begin + p];
      const CkptK K = ckpt_level(P, l, c, ke);
      const ZeroK Z = zero_level(P, z);
      const double rw = rr[iw], rg = rr[ig];
      const WoGoK W = wogo_levels(P, Z, rw, om[iw], rg, om[ig]);
      // Exact frontier: lower bounds of the optimizer level's peak and first-microbatch extras over
      // the strip's optimizer ratios, then a first candidate bound for the whole strip.  Every
      // input of the level is non-negative, so each of its operations is non-decreasing in the
      // ratio r or in 1 - r; the bounds repeat the level's own operations on the smallest r and
      // the smallest 1 - r (the resident states shrink with r, the offloaded states' buffer and
      // the extras grow with it), and rounding to nearest is monotone: each is at most the value
      // of every optimizer ratio, the peak's as max(forward, backward) of two lower bounds.
      [[maybe_unused]] double Bmin = 0.0, Hxmin = 0.0, Dxmin = 0.0;
      if constexpr (BLK) {
        const double base = __builtin_fma(q_lo, Z.So, W.Swg) + W.Wbuf;
        const double BF = (base + __builtin_fma(r_lo, Z.Obo, W.Og)) + P.Xd;
        const double BB = ((base + W.Gbuf) + K.Rc) + P.Xd;
        Bmin = __builtin_fmax(BF, BB);
        Hxmin = __builtin_fma(r_lo, Z.So, W.DG) * iP;
        Dxmin = __builtin_fma(r_lo, Z.So, W.DW) * iP;
        {
          // The strip bound, before the stable times: with every slowdown factor at least 1 a
          // stable time is at least each of its streams' times (compute, GPU-GPU and the host
          // streams, whose smallest values come with the smallest activation ratio), and the
          // stash and offload buffers are at least fma(r_lo, 2A, q_lo * KA).  The bound is the
          // block bound below with those values in place of the block's own, so it is at most
          // every configuration's; a strip that fails in every lane of the wave is skipped whole
          // (the relative 2^-30 covers the rounding of the stable time as well).
          const double hsl = __builtin_fma(r_lo, K.A, W.HW) * iP, dsl = __builtin_fma(r_lo, K.A, W.DG) * iP;
          const double mem = Bmin + __builtin_fma(r_lo, P.A2, q_lo * K.KA);
          const unsigned int j0 = (unsigned int)__builtin_fmin(mem * kNB, 63.0);
          const double pm = *reinterpret_cast<const double*>(
              reinterpret_cast<const char*>(s_filt[wave]) + __umul24(j0, (unsigned int)sizeof(FiltEntry)));
          const double tl = __builtin_fmax(__builtin_fmax(K.C, Z.G2Gs), __builtin_fmax(hsl, dsl));
          const double lb = __builtin_fma(Gd - 1.0, tl, __builtin_fmax(hsl + Hxmin, dsl + Dxmin));
          if (!__builtin_amdgcn_ballot_w64((mem <= M) & (lb * (1.0 - 0x1p-30) < pm))) continue;
        }
      }

      // First microbatch: every configuration of the strip with a non-zero offload ratio
      // starts with compute, both host streams and (if it carries traffic) GPU-GPU.
      const int pat1 = Z.G2Gf > 0.0 ? 15 : 13;
      const KnownRow fr = known_row(tab, pat1, K.C, Z.G2Gf);
      const bool zero_strip = r0_zero && rw == 0.0 && rg == 0.0;
      // First-microbatch time of the strip's all-zero configuration (no host streams).
      const double T1z = interference_zero(K.C, Z.G2Gf, tab);
      s_oo[tid] = oo_inputs(P, K, Z, W);
      const double A = K.A, KA = K.KA, A2 = P.A2, HW = W.HW, DG = W.DG;
      // Block bound: the strip's smallest optimizer-level peak and first-microbatch extras over
      // the optimizer ratios, each the minimum of the values the configurations use.
      const unsigned int lid_strip = (unsigned int)s * (unsigned int)R2;
      // With a positive activation ratio both host streams run, so the stable microbatch's
      // first round has the pattern compute + both host streams (+ GPU-GPU when it carries
      // traffic).
      const int pats = Z.G2Gs > 0.0 ? 15 : 13;

      // Activation ratios in blocks of IB: the values a block keeps across the optimizer
      // ratios fit the registers, at the price of one more optimizer-level evaluation per
      // block.  A block's stable times, and per optimizer ratio its first-microbatch times, are
      // formed before its memory, objective and reduction steps, so that the interference rounds
      // of its configurations are straight-line code.
#pragma unroll
      for (int ib = 0; ib < R; ib += IB) {
        // Stable time per activation ratio (it does not depend on the optimizer ratio).
        const int nb = R - ib < IB ? R - ib : IB;  // configurations of the block
        const KnownRow sr = known_row(tab, pats, K.C, Z.G2Gs);
        double tt[IB];
        [[maybe_unused]] int fst[IB];  // dump variant: the form of each stable time
        [[maybe_unused]] double hsmin = 0.0, dsmin = 0.0;  // block bound: the smallest host streams
        {
          double hs[IB], ds[IB];
          bool fs[IB];
#pragma unroll
          for (int c = 0; c < IB; ++c) {
            const int ia = ib + c;
            if (ia >= R) break;
            hs[c] = __builtin_fma(rr[ia], K.A, W.HW) * iP;
            ds[c] = __builtin_fma(rr[ia], K.A, W.DG) * iP;
            fs[c] = ia == 0 && r0_zero;
          }
          interference_known_n<IB>(sr, hs, ds, fs, tt, fst, nb, tab, RK);
          if constexpr (BLK) {
            hsmin = hs[0];
            dsmin = ds[0];
#pragma unroll
            for (int c = 1; c < IB; ++c) {
              if (ib + c >= R) break;
              hsmin = __builtin_fmin(hsmin, hs[c]);
              dsmin = __builtin_fmin(dsmin, ds[c]);
            }
          }
          // Activation ratio 0 leaves the host streams to the weights and gradients alone: the
          // first round's pattern is not known in advance.
          if (ib == 0 && r0_zero) {
            tt[0] = interference(K.C, Z.G2Gs, hs[0], ds[0], tab);
            fst[0] = kFormGeneric;
          }
        }
        // Weight samples: the block's smallest stable time, for the lower bound below.
        [[maybe_unused]] double t_min = tt[0];
        if constexpr (AL) {
#pragma unroll
          for (int c = 1; c < IB; ++c)
            if (ib + c < R) t_min = __builtin_fmin(t_min, tt[c]);
        }

        if constexpr (BLK) {
          // Exact frontier: the candidate bound of the configurations below, taken once for the
          // block.  Each of its terms is at most, over the block's optimizer and activation
          // ratios, the value a configuration's bound uses (its memory from the peak's bound and
          // the smallest stash, its host streams from the smallest stable parts and the extras'
          // bounds, the smallest stable time); rounding is monotone, so the block's memory,
          // bucket estimate and bound are at most each configuration's, and its threshold pm at
          // least each one's (pm does not increase with the bucket).  A block that fails in every lane of the wave holds no
          // configuration that passes its own bound, and none that can be a candidate: the
          // strip's all-zero configuration, whose time is formed without the bound, has host
          // streams 0 and so an objective of at least (G - 1) t as well.
          double tmin = tt[0], somin = __builtin_fma(rr[ib], A2, om[ib] * KA);
#pragma unroll
          for (int c = 1; c < IB; ++c) {
            if (ib + c >= R) break;
            tmin = __builtin_fmin(tmin, tt[c]);
            somin = __builtin_fmin(somin, __builtin_fma(rr[ib + c], A2, om[ib + c] * KA));
          }
          const double mem = Bmin + somin;
          const unsigned int j0 = (unsigned int)__builtin_fmin(mem * kNB, 63.0);
          const double pm = *reinterpret_cast<const double*>(
              reinterpret_cast<const char*>(s_filt[wave]) + __umul24(j0, (unsigned int)sizeof(FiltEntry)));
          const double lb = __builtin_fma(Gd - 1.0, tmin, __builtin_fmax(hsmin + Hxmin, dsmin + Dxmin));
          if (!__builtin_amdgcn_ballot_w64((mem <= M) & (lb * (1.0 - 0x1p-30) < pm))) continue;
        }

#pragma unroll 1
        for (int io = 0; io < R; ++io) {
          const OoK O = oo_level(s_oo[tid], rr[io], om[io], iP);
          const bool zero_oo = zero_strip && io == 0;
          const unsigned int lid_oo = lid_strip + (unsigned int)(io * R);
          [[maybe_unused]] double dn_blk[AL ? IB : 1];  // weight samples: the block's deltas (NaN
                                                        // when infeasible)
          double T1b[IB];
          [[maybe_unused]] int f1b[IB];  // dump variant: the form of each first-microbatch time
          {
            double hf[IB], df[IB];
            bool fz[IB];
#pragma unroll
            for (int c = 0; c < IB; ++c) {
              const int ia = ib + c;
              if (ia >= R) break;
              hf[c] = __builtin_fma(rr[ia], A, HW) * iP + O.H2Dx;
              df[c] = __builtin_fma(rr[ia], A, DG) * iP + O.D2Hx;
              fz[c] = ia == 0 && zero_oo;
              if constexpr (EX) {
                // The exact frontier's candidates are feasible and below every lower bucket's
                // minimum pm of their bucket; a configuration that fails either needs no
                // first-microbatch time (its candidate test fails).  With every slowdown factor
                // at least 1 each stream's standalone time is progressed by at most the phase
                // length in every round, so T1 is at least every stream's time, in particular
                // max(H2D, D2H), and obj = G t + (T1 - t) >= (G - 1) t + max(H2D, D2H); the
                // bound is lowered by a relative 2^-30, far above the rounding of either side (a
                // few dozen operations of relative error 2^-53), so a configuration whose bound
                // is not below pm cannot be a candidate.  (Compute and GPU-GPU would tighten it
                // little and cost registers: 92 against 72 bytes of scratch, same time.)  pm does
                // not increase with the bucket (a prefix minimum), so the estimate
                // j0 = floor(mem * kNB) <= j of the bucket step serves: pm[j0] >= pm[j].
                const double mem = O.Bmax + __builtin_fma(rr[ia], A2, om[ia] * KA);
                const unsigned int j0 = (unsigned int)__builtin_fmin(mem * kNB, 63.0);
                const double pm = *reinterpret_cast<const double*>(
                    reinterpret_cast<const char*>(s_filt[wave]) + __umul24(j0, (unsigned int)sizeof(FiltEntry)));
                const double lb = __builtin_fma(Gd - 1.0, tt[c], __builtin_fmax(hf[c], df[c]));
                // Such a lane takes no part in the choice of form; its T1, and so its objective,
                // is NaN, which fails the candidate test.
                fz[c] = fz[c] | !((mem <= M) & (lb * (1.0 - 0x1p-30) < pm));
              }
            }
            interference_known_n<IB, EX>(fr, hf, df, fz, T1b, f1b, nb, tab, RK);
          }
#pragma unroll
          for (int c = 0; c < IB; ++c) {
            const int ia = ib + c;
            if (ia >= R) break;
            const double ra = rr[ia];
            const double SO = __builtin_fma(ra, A2, om[ia] * KA);  // stash + offload buffers
            const double mem = O.Bmax + SO;
            double T1 = T1b[c];
            if (ia == 0) T1 = zero_oo ? T1z : T1;
            // Exact frontier: a lane whose time was not formed (NaN) cannot hold a candidate, and
            // when no lane of the wave has a time the configuration is done.
            if constexpr (EX) {
              if (!__builtin_amdgcn_ballot_w64(T1 == T1)) continue;
            }
            const double tv = tt[c];
            const double d = T1 - tv;
            const double obj = __builtin_fma(Gd, tv, d);

            // Bucket j = min{j : mem <= E_j}: floor(mem * kNB) is j or j - 1 (kNB carries a
            // 2^-40 margin), so one comparison with E settles it.  An infeasible
            // configuration (Eq. 4: mem > M = E_{NB-1}) has floor(mem * kNB) >= NB - 1 and
            // lands on a sink: past NB - 1 the edges are +inf.  j0 = j - 1 needs mem within a
            // relative 2^-40 above an edge, or an infeasible mem just above M: rare, so only
            // entry j0's edge and key are read, and entry j0 + 1 (<= 64: entry 64's edge is
            // +inf) only by lanes whose mem exceeds E_j0.
            const int j0 = (int)__builtin_fmin(mem * kNB, 64.0);
            const unsigned int off0 = __umul24((unsigned int)j0, (unsigned int)sizeof(BucketEntry));
            char* const b0 = reinterpret_cast<char*>(bucket) + off0;
            wave_sync();  // read the entry after every earlier update of the wave
            const double e0 = reinterpret_cast<const BucketEntry*>(b0)->edge;
            const unsigned long long k_lo = reinterpret_cast<const BucketEntry*>(b0)->key;
            if constexpr (DM) {
              double* o = a.dump + kDumpWords * (a.dump_off[x] + (int64_t)(s - tile.strip_begin) * R2 + io * R + ia);
              o[0] = tv;
              o[1] = d;
              o[2] = mem;
              o[3] = obj;
              o[4] = (double)(j0 + (mem > e0 ? 1 : 0));
              o[5] = (double)((ia == 0 && zero_oo ? kFormZero : f1b[c]) + 8 * fst[c]);
              continue;
            }
            if constexpr (EX) {
              // Exact frontier candidates: feasible, below every lower bucket's minimum, and not
              // dominated by the bucket's winner (no more memory and no smaller objective, not
              // both equal).  Every frontier point passes; the scan after the sort decides.
              const int j = min(j0 + (mem > e0 ? 1 : 0), 63);
              const FiltEntry f = s_filt[wave][j];
              const bool cand = (mem <= M) & (obj < f.pm) &
                                !(((obj > f.bobj) & (mem >= f.bmem)) | ((obj >= f.bobj) & (mem > f.bmem)));
              const unsigned long long m = __builtin_amdgcn_ballot_w64(cand);
              if (!m) continue;
              int64_t slot = 0;
              if (cand) {
                const unsigned int below = __builtin_amdgcn_mbcnt_hi(
                    (unsigned int)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)m, 0u));
                slot = n_cand + below;
                if (slot < n_end) {
                  a.cand_key[slot] = (unsigned long long)__double_as_longlong(mem);
                  a.cand_obj[slot] = obj;
                  a.cand_id[slot] = g.base + (uint64_t)(lid_oo + (unsigned int)ia);
                }
              }
              // Past the window: the overflow pool, in chunks of kPoolChunk slots per wave (one
              // device-wide atomic per chunk), else counted only and the tile is evaluated again.
              const bool over = cand && slot >= n_end;
              const unsigned long long mo = __builtin_amdgcn_ballot_w64(over);
              if (mo && a.pool_count) {
                const int k = __builtin_popcountll(mo);
                if (pool_used + k > kPoolChunk) {
                  pool_holes(a, pool_base, pool_used, lane);
                  const int leader = __builtin_ctzll(mo);
                  unsigned long long b = 0;
                  if (lane == leader) b = atomicAdd(a.pool_count, (unsigned long long)kPoolChunk);
                  const unsigned long long bb = __shfl(b, leader, 64);
                  pool_base = ((unsigned long long)__builtin_amdgcn_readfirstlane((unsigned int)(bb >> 32)) << 32) |
                              (unsigned long long)__builtin_amdgcn_readfirstlane((unsigned int)bb);
                  pool_used = 0;
                }
                if (over) {
                  const unsigned long long pos = pool_base + (unsigned long long)pool_used + __builtin_amdgcn_mbcnt_hi(
                      (unsigned int)(mo >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)mo, 0u));
                  if (pos < (unsigned long long)a.pool_cap) {
                    a.pool_key[pos] = (unsigned long long)__double_as_longlong(mem);
                    a.pool_obj[pos] = obj;
                    a.pool_id[pos] = g.base + (uint64_t)(lid_oo + (unsigned int)ia);
                    a.pool_tile[pos] = t;
                    a.pool_rank[pos] = (int32_t)(slot - n_beg);
                  } else {
                    dropped = true;
                  }
                }
                pool_used += k;
              } else if (mo) {
                dropped = dropped | over;
              }
              n_cand += __builtin_popcountll(m);
              continue;
            }
            const bool up = mem > e0;

            // Lexicographic (obj, id) minimum per bucket without a serial loop: the lanes
            // that beat their bucket's entry lower the objective bits with an LDS atomic
            // minimum; a lane that sees its bucket's objective drop clears the id, then the
            // lanes whose objective equals the new minimum lower the id.  The LDS operations
            // of a wave execute in program order and each step addresses the same words as
            // the one before, so each step sees the previous one's result.
            const unsigned long long key = (unsigned long long)__double_as_longlong(obj);
            // A candidate beats the entry: key < k_old, or an equal key with a lower id.  No
            // lane with key > k_old is one, so the exact test waits for a lane with key <= k_old
            // or a lane in entry j0 + 1 (combined as wave masks by the scalar ALU).
            const unsigned long long m_up = __builtin_amdgcn_ballot_w64(up);
            const unsigned long long m_lo = __builtin_amdgcn_ballot_w64(key <= k_lo);
            if (m_lo | m_up) {
              BucketEntry* const be = reinterpret_cast<BucketEntry*>(b0 + (up ? sizeof(BucketEntry) : 0));
              const unsigned long long k_old = up ? lds_load(&be->key) : k_lo;
              const unsigned int lid = lid_oo + (unsigned int)ia;
              const unsigned int i_old = lds_load(&be->lid);
              const bool cand = (key < k_old) | ((key == k_old) & (lid < i_old));
              if (cand) atomicMin(&be->key, key);
              const unsigned long long k_new = cand ? lds_load(&be->key) : 0ull;
              if (cand && k_new < k_old) lds_store(&be->lid, 0xFFFFFFFFu);
              if (cand && key == k_new) atomicMin(&be->lid, lid);
            }

            if constexpr (AL) dn_blk[c] = mem <= M ? d : __builtin_nan("");
          }

          if constexpr (AL) {
            // Eq. 4 for every weight sample, feasible configurations only: an infeasible one
            // carries a NaN delta, so each of its weighted values is NaN and compares false.
            // First the block's configurations against every sample's entry as it stands (no
            // lane can beat an entry it does not beat now: entries only decrease), each
            // sample's values read once for the block; the exact sequence only when some lane
            // of the wave may win.  All lanes address the sample's single entry; the same
            // three-step LDS sequence as the buckets' keeps the lexicographic minimum.
            //
            // Before that, one bound per sample and block: with a = alpha*G >= 0 and
            // b = 1 - alpha >= 0, fma(a, t, b*d) is non-decreasing in t and d under rounding to
            // nearest, so fma(a, t_min, b*d_min) over the block's smallest t and smallest
            // feasible d is at most every feasible configuration's value.  A sample whose bound
            // exceeds its entry on every lane cannot be won by the block, and its per-
            // configuration values are not formed (NaN deltas drop out of the minimum; a block
            // without a feasible configuration has a NaN bound, which compares false).
            wave_sync();
            double d_min = dn_blk[0];
#pragma unroll
            for (int c = 1; c < IB; ++c)
              if (ib + c < R) d_min = __builtin_fmin(d_min, dn_blk[c]);
            unsigned int qmask = 0;  // samples some lane of the wave may win
#pragma unroll 1
            for (int q = 0; q < a.n_alpha; ++q) {
              const double2 ab = s_ab[wave][q];
              const double cur = lds_load(&s_aent[wave][q].val);
              if (!__builtin_amdgcn_ballot_w64(__builtin_fma(ab.x, t_min, ab.y * d_min) <= cur)) continue;
              bool any = false;
#pragma unroll
              for (int c = 0; c < IB; ++c) {
                if (ib + c >= R) break;
                any = any | (__builtin_fma(ab.x, tt[c], ab.y * dn_blk[c]) <= cur);
              }
              if (__builtin_amdgcn_ballot_w64(any)) qmask |= 1u << q;
            }
            if (qmask) {
#pragma unroll 1
              for (unsigned int qs = qmask; qs; qs &= qs - 1) {
                const int q = __builtin_ctz(qs);
                const double2 ab = s_ab[wave][q];
                AlphaEntry* const e = &s_aent[wave][q];
#pragma unroll
                for (int c = 0; c < IB; ++c) {
                  const int ia = ib + c;
                  if (ia >= R) break;
                  const double v = __builtin_fma(ab.x, tt[c], ab.y * dn_blk[c]);
                  wave_sync();
                  const double cur = lds_load(&e->val);
                  if (__builtin_amdgcn_ballot_w64(v <= cur)) {
                    const unsigned int lid = lid_oo + (unsigned int)ia;
                    const unsigned long long ak = order_key(v);
                    const unsigned long long ak_old = lds_load(&e->key);
                    const unsigned int ai_old = lds_load(&e->lid);
                    const bool cand = (v <= cur) & ((ak < ak_old) | ((ak == ak_old) & (lid < ai_old)));
                    if (cand) atomicMin(&e->key, ak);
                    const unsigned long long ak_new = cand ? lds_load(&e->key) : 0ull;
                    if (cand && ak_new < ak_old) lds_store(&e->lid, 0xFFFFFFFFu);
                    if (cand && ak == ak_new) {
                      atomicMin(&e->lid, lid);
                      lds_store(&e->val, v);
                    }
                  }
                }
              }
            }
          }
        }
      }
    }
    // The tile's partials: lane j = bucket j.
    if constexpr (DM) {
    } else if constexpr (EX) {
      // The wave's pool chunk is updated inside the strip loop, which lanes past a ragged
      // tile's last strip leave early: lane 0 stays to the end and holds the current chunk.
      {
        const unsigned long long b = __shfl(pool_base, 0, 64);
        pool_base = ((unsigned long long)__builtin_amdgcn_readfirstlane((unsigned int)(b >> 32)) << 32) |
                    (unsigned long long)__builtin_amdgcn_readfirstlane((unsigned int)b);
        pool_used = __builtin_amdgcn_readfirstlane(__shfl(pool_used, 0, 64));
      }
      // Saturated at 2^31 - 1, which the host rejects (no tile of a space with fewer than
      // 2^32 candidates reaches it).
      if (lane == 0) a.cnt_tile[t] = (int32_t)min(n_cand - n_beg, (int64_t)0x7FFFFFFF);
      const unsigned long long md = __builtin_amdgcn_ballot_w64(dropped);
      if (lane == 0 && a.tile_drop) a.tile_drop[t] = md ? 1 : 0;
    } else {
      wave_sync();
      const unsigned int bl = bucket[lane].lid;
      a.part_obj[(size_t)t * 64 + lane] = __longlong_as_double((long long)bucket[lane].key);
      a.part_id[(size_t)t * 64 + lane] = bl == 0xFFFFFFFFu ? kNone : g.base + (uint64_t)bl;
    }
    if constexpr (AL) {
      if (lane < a.n_alpha) {
        const AlphaEntry e = s_aent[wave][lane];
        a.part_aobj[(size_t)t * a.n_alpha + lane] = e.val;
        a.part_aid[(size_t)t * a.n_alpha + lane] = e.lid == 0xFFFFFFFFu ? kNone : g.base + (uint64_t)e.lid;
      }
    }
    if (!claims) break;
    for (;;) {
      int c = 0;
      if (lane == 0) c = atomicAdd(a.work + counter * kCounterStride, 1);
      c = __builtin_amdgcn_readfirstlane(__shfl(c, 0, 64));
      const int64_t next = (int64_t)n_waves + counter + (int64_t)kClaimCounters * c;
      if (next < n_items) {
        x = (int)next;
        break;
      }
      if (++exhausted == kClaimCounters) {  // every counter has run out: no item is left
        x = n_items;
        break;
      }
      counter = counter + 1 == kClaimCounters ? 0 : counter + 1;
    }
  }
  if constexpr (EX) {
    if (a.pool_count) pool_holes(a, pool_base, pool_used, lane);
  }
}

// ---------------------------------------------------------------------------------------
// K2: lane j owns bucket j.  With W = 4, a block of four waves per group: each wave takes
// the lexicographic minimum over every fourth tile of the group (its full-size ones, then its
// small ones), so the largest group's chain of dependent loads is a quarter as long, and the
// first wave combines the four in LDS; with W = 1 (spaces whose groups hold few tiles), a wave
// per group.  Then the group's best by a butterfly over the 64 lanes and the staircase by an
// exclusive prefix minimum over the buckets.
// ---------------------------------------------------------------------------------------
template <int kW>
__global__ __launch_bounds__(256) void k_reduce(ReduceArgs a) {
  __shared__ double s_o[kW][64];
  __shared__ uint64_t s_i[kW][64];
  __shared__ double s_ao[kW][kMaxAlphas];
  __shared__ uint64_t s_ai[kW][kMaxAlphas];
  const int lane = threadIdx.x & 63;
  // Wave-uniform (stated, so that the group record arrives by scalar loads and the tile loops
  // run on scalar registers).
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wave = kW > 1 ? wv : 0;  // the wave's share of the tiles
  const int64_t g = kW > 1 ? (int64_t)blockIdx.x : (int64_t)blockIdx.x * 4 + wv;
  if (g >= a.n_groups) return;
  const DevGroup grp = load_uniform(a.groups + g);
  double obj = __builtin_huge_val();
  uint64_t id = kNone;
  if (lane < a.NB) {  // several tiles' loads in flight
#pragma unroll 4
    for (int t = grp.tile_begin + wave; t < grp.tile_begin + grp.n_tiles; t += kW) {
      const double o = __builtin_nontemporal_load(a.part_obj + (size_t)t * 64 + lane);  // read once
      const uint64_t i = __builtin_nontemporal_load(a.part_id + (size_t)t * 64 + lane);
      if (lex_less(o, i, obj, id)) {
        obj = o;
        id = i;
      }
    }
#pragma unroll 4
    for (int t = grp.tail_begin + wave; t < grp.tail_begin + grp.n_tail; t += kW) {
      const double o = __builtin_nontemporal_load(a.part_obj + (size_t)t * 64 + lane);
      const uint64_t i = __builtin_nontemporal_load(a.part_id + (size_t)t * 64 + lane);
      if (lex_less(o, i, obj, id)) {
        obj = o;
        id = i;
      }
    }
  }
  if constexpr (kW > 1) {
    s_o[wave][lane] = obj;
    s_i[wave][lane] = id;
  }
  double ao = __builtin_huge_val();
  uint64_t ai = kNone;
  if (lane < a.n_alpha) {  // lane a: weight sample a
    for (int t = grp.tile_begin + wave; t < grp.tile_begin + grp.n_tiles; t += kW) {
      const double o = a.part_aobj[(size_t)t * a.n_alpha + lane];
      const uint64_t i = a.part_aid[(size_t)t * a.n_alpha + lane];
      if (lex_less(o, i, ao, ai)) {
        ao = o;
        ai = i;
      }
    }
    for (int t = grp.tail_begin + wave; t < grp.tail_begin + grp.n_tail; t += kW) {
      const double o = a.part_aobj[(size_t)t * a.n_alpha + lane];
      const uint64_t i = a.part_aid[(size_t)t * a.n_alpha + lane];
      if (lex_less(o, i, ao, ai)) {
        ao = o;
        ai = i;
      }
    }
    if constexpr (kW > 1) {
      s_ao[wave][lane] = ao;
      s_ai[wave][lane] = ai;
    }
  }
  if constexpr (kW > 1) {
    __syncthreads();
    if (wave != 0) return;
    // The group's lexicographic minima over the waves' (order does not matter).
#pragma unroll
    for (int w = 1; w < kW; ++w)
      if (lex_less(s_o[w][lane], s_i[w][lane], obj, id)) {
        obj = s_o[w][lane];
        id = s_i[w][lane];
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
  if (lane < a.n_alpha) {
#pragma unroll
    for (int w = 1; w < kW; ++w)
      if (lex_less(s_ao[w][lane], s_ai[w][lane], ao, ai)) {
        ao = s_ao[w][lane];
        ai = s_ai[w][lane];
      }
    a.alpha_obj[g * a.n_alpha + lane] = ao;
    a.alpha_id[g * a.n_alpha + lane] = ai;
  }
}

// ---------------------------------------------------------------------------------------
// Per-id evaluation with the same level functions (parity and result extraction).
// ---------------------------------------------------------------------------------------
struct OneVal {
  double t, d, mem, obj;
};

// One configuration by id: binary search of the group, mixed-radix decode, and the level
// functions of the evaluation kernel.
__device__ OneVal eval_one(const EvalArgs& a, uint64_t id) {
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
  const double* tab = &hw.itab[0][0];
  const PairK P = pair_level(a.m, g.PP, g.k, g.l, a.pairs[g.pair_begin + p], hw);
  const CkptK K = ckpt_level(P, g.l, c, ke);
  const ZeroK Z = zero_level(P, z);
  const WoGoK W = wogo_levels(P, Z, r[iw], om[iw], r[ig], om[ig]);
  const OoK O = oo_level(oo_inputs(P, K, Z, W), r[io], om[io], hw.iP);
  const double ra = r[ia];
  const double SO = __builtin_fma(ra, P.A2, om[ia] * K.KA);
  const double H2Ds = __builtin_fma(ra, K.A, W.HW) * hw.iP;
  const double D2Hs = __builtin_fma(ra, K.A, W.DG) * hw.iP;
  OneVal res;
  res.mem = O.Bmax + SO;
  res.t = interference<kTabStride>(K.C, Z.G2Gs, H2Ds, D2Hs, tab);
  const double T1 = interference<kTabStride>(K.C, Z.G2Gf, H2Ds + O.H2Dx, D2Hs + O.D2Hx, tab);
  res.d = T1 - res.t;
  res.obj = __builtin_fma((double)g.G, res.t, res.d);
  return res;
}

__global__ __launch_bounds__(256) void k_eval_ids(EvalArgs a, const uint64_t* __restrict__ ids,
                                                  int64_t n, double* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const OneVal v = eval_one(a, ids[i]);
  out[4 * i + 0] = v.t;
  out[4 * i + 1] = v.d;
  out[4 * i + 2] = v.mem;
  out[4 * i + 3] = v.obj;
}

// Live tiles of the exact frontier: one wave per tile, lane j = bucket j.  A candidate needs an
// objective below every lower bucket's minimum (pm); the tile's partial for bucket j is the
// minimum objective of its configurations in that bucket, so a tile none of whose partials is
// below its pm holds no candidate.
__global__ __launch_bounds__(kReduceBlock) void k_live(EvalArgs a, const FiltEntry* __restrict__ filt,
                                                      uint8_t* __restrict__ live) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (kReduceBlock / 64) + (threadIdx.x >> 6);
  if (t >= a.n_tiles) return;
  const int64_t g = a.tiles[t].group;
  const bool may = lane < a.NB && a.part_obj[t * 64 + lane] < filt[g * 64 + lane].pm;
  const unsigned long long m = __builtin_amdgcn_ballot_w64(may);
  if (lane == 0) live[t] = m != 0ull ? 1 : 0;
}

// Candidate filter of the exact frontier: one wave per group, lane j = bucket j.
__global__ __launch_bounds__(kReduceBlock) void k_filter(EvalArgs a, const double* __restrict__ bucket_obj,
                                                         const uint64_t* __restrict__ bucket_id,
                                                         FiltEntry* __restrict__ filt) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * (kReduceBlock / 64) + (threadIdx.x >> 6);
  if (g >= a.n_groups) return;
  const double obj = lane < a.NB ? bucket_obj[g * 64 + lane] : __builtin_huge_val();
  const uint64_t id = lane < a.NB ? bucket_id[g * 64 + lane] : kNone;
  double pm = obj;  // inclusive prefix minimum over buckets 0..lane
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(pm, off, 64);
    if (lane >= off) pm = __builtin_fmin(pm, o);
  }
  double below = __shfl_up(pm, 1, 64);
  if (lane == 0) below = __builtin_huge_val();
  FiltEntry f;
  f.pm = below;
  f.bobj = obj;
  f.bmem = id == kNone ? __builtin_huge_val() : eval_one(a, id).mem;
  filt[g * 64 + lane] = f;
}

int check_launch() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

template <int R, int MODE>
void launch_eval_rm(const EvalArgs& a, int blocks, hipStream_t st) {
  hipLaunchKernelGGL((k_eval<R, MODE>), dim3(blocks), dim3(kBlock), 0, st, a, a.ratio, (const PairK*)a.pk);
}

template <int R>
void launch_eval_r(const EvalArgs& a, int blocks, int mode, hipStream_t st) {
  switch (mode) {
    case kModeAlpha: launch_eval_rm<R, kModeAlpha>(a, blocks, st); break;
    case kModeEmit: launch_eval_rm<R, kModeEmit>(a, blocks, st); break;
    case kModeDump: launch_eval_rm<R, kModeDump>(a, blocks, st); break;
    default: launch_eval_rm<R, kModeBuckets>(a, blocks, st); break;
  }
}

template <int R, int MODE>
int blocks_per_cu_rm() {
  int n = 0;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_eval<R, MODE>, kBlock, 0) == hipSuccess ? n : 1;
}

template <int R>
int blocks_per_cu_r(int mode) {
  switch (mode) {
    case kModeAlpha: return blocks_per_cu_rm<R, kModeAlpha>();
    case kModeEmit: return blocks_per_cu_rm<R, kModeEmit>();
    case kModeDump: return blocks_per_cu_rm<R, kModeDump>();
    default: return blocks_per_cu_rm<R, kModeBuckets>();
  }
}

#define MIST_FOR_EACH_R(X) \
  X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16)

}  // namespace

int eval_blocks_per_cu(int R, int mode) {
  switch (R) {
#define MIST_CASE(n) \
  case n:            \
    return blocks_per_cu_r<n>(mode);
    MIST_FOR_EACH_R(MIST_CASE)
#undef MIST_CASE
    default:
      return 1;
  }
}

int launch_eval(const EvalArgs& a, int blocks, int mode, void* stream) {
  if (a.n_tiles <= 0) return 0;
  hipStream_t st = (hipStream_t)stream;
  switch (a.R) {
#define MIST_CASE(n)                       \
  case n:                                  \
    launch_eval_r<n>(a, blocks, mode, st); \
    break;
    MIST_FOR_EACH_R(MIST_CASE)
#undef MIST_CASE
    default:
      return (int)hipErrorInvalidValue;
  }
  return check_launch();
}

int launch_pairs(const EvalArgs& a, void* stream) {
  if (a.n_pk <= 0) return 0;
  hipLaunchKernelGGL(k_pairs, dim3((unsigned)((a.n_pk + 255) / 256)), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch();
}

int launch_reduce(const ReduceArgs& a, void* stream) {
  if (a.n_groups <= 0) return 0;
  // Four waves per group pay off when some group's tiles make a long chain of loads and the
  // groups are few enough that the idle waves of small groups cost little (measured: 23 ->
  // 14 us on gpt2.7b-d16, 44 -> 31 us on llama13b-d64; 89 -> 93 us on llama42b-d128-hw64,
  // 66,496 groups, which keeps a wave per group).
  if (a.max_group_tiles >= 16 && a.n_groups <= 16384)
    hipLaunchKernelGGL(k_reduce<4>, dim3((unsigned)a.n_groups), dim3(256), 0, (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(k_reduce<1>, dim3((unsigned)((a.n_groups + 3) / 4)), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch();
}

int launch_live(const EvalArgs& a, const FiltEntry* filt, uint8_t* live, void* stream) {
  if (a.n_tiles <= 0) return 0;
  const int per = kReduceBlock / 64;
  const int64_t blocks = ((int64_t)a.n_tiles + per - 1) / per;
  hipLaunchKernelGGL(k_live, dim3((unsigned)blocks), dim3(kReduceBlock), 0, (hipStream_t)stream, a, filt, live);
  return check_launch();
}

int launch_filter(const EvalArgs& a, const double* bucket_obj, const uint64_t* bucket_id, FiltEntry* filt,
                  void* stream) {
  if (a.n_groups <= 0) return 0;
  const int per = kReduceBlock / 64;
  const int64_t blocks = (a.n_groups + per - 1) / per;
  hipLaunchKernelGGL(k_filter, dim3((unsigned)blocks), dim3(kReduceBlock), 0, (hipStream_t)stream, a, bucket_obj,
                     bucket_id, filt);
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
