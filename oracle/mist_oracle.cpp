// Mist intra-stage tuner: plain single-threaded CPU oracle.
//
// TEST INFRASTRUCTURE ONLY.  This file is the reference that the GPU path is
// checked against.  Only the tests, the smoke check and the benchmark's CPU
// baseline may build, load or call it; the product path never does.  It shares
// no code, header, table or helper with the HIP library: descriptor layouts are
// re-declared here as plain data.
//
// What it computes (Zhu et al., "Mist", EuroSys'25):
//   * the configuration space of one pipeline stage: the per-stage tuple of
//     Sec. 5.1 / Table 2 (b, DP, TP, ZeRO, CKPT, WO, GO, OO, AO) for every
//     candidate stage (G, PP, in-flight count, layer count) that intra-stage
//     tuning is asked about (Sec. 5.3, Eq. 4, and the IntraStagePareto query of
//     Eq. 3);
//   * for every configuration, the stage's peak memory (the constraint of
//     Eq. 4), its stable-microbatch time t and first-microbatch delta d
//     (Eq. 5-6) through the interference model of Algorithm 1 (Sec. 5.2.2);
//   * per group, the feasible minimum of G*t + d (Eq. 4 at alpha = 1/2, scaled
//     by 2), with the lowest configuration id breaking ties, per memory-budget
//     bucket and overall, and the bucketed time-vs-memory staircase.
//
// The paper derives its cost expressions by symbolic tracing, liveness analysis
// and a profiled operator database (Sec. 5.2.1), none of which is printed.  The
// expressions below are this project's written-out cost model (ZeRO's K = 12
// state accounting, Korthikanti et al.'s activation accounting, Megatron's
// FLOP formula, ring-collective byte counts), evaluated in the nested-loop
// order of the tuple so that each quantity is computed at the loop level whose
// digits it depends on.  Every floating-point operation is listed explicitly;
// compile with -ffp-contract=off and without fast-math.  fma() is used exactly
// where the cost model says so, and nowhere else.
//
// The arithmetic is written once as templates over the number type R so that a
// counting build (R = Counted) reports the FP64 operations of the definition
// per configuration: add, sub and mul count 1, fma counts 2, min/max/compare 0.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <vector>

namespace {

// ---------------------------------------------------------------------------
// Descriptors (plain data; same field order as the C-ABI descriptors).
// ---------------------------------------------------------------------------
struct Model {
  int32_t arch;  // 0 = GPT (LayerNorm, GeLU MLP f, learned positions), 1 = LLAMA (RMSNorm, SwiGLU f)
  int32_t n_layers;
  int64_t hidden;
  int32_t heads;
  int32_t kv_heads;
  int64_t ffn;
  int64_t seq;
  int64_t vocab;
  int32_t bytes_w;    // bytes per fp16/bf16 weight, gradient and activation element
  int32_t bytes_opt;  // bytes of fp32 master + Adam m + v per parameter (ZeRO's K)
  int32_t flash;      // 1 = FlashAttention (no stored softmax)
};

struct Hw {
  double flops;      // peak FLOP/s
  double mem_bytes;  // memory budget (bytes)
  double pcie_bw;    // CPU<->GPU bytes/s
  double link_bw;    // GPU<->GPU bytes/s
  double eta_max;    // asymptotic compute efficiency
  double n_half;     // tokens at which efficiency is half of eta_max
  double phi[16][4]; // slowdown factors, [co-running mask][stream]
  double eta_tab[16];  // with eta_max == 0: measured compute efficiency of the space's i-th
                       // microbatch size (the operator database of Sec. 5.2.1)
};

struct Space {
  int64_t n_devices;
  int64_t global_batch;
  const int32_t* mb;
  int32_t n_mb;
  const double* ratios;
  int32_t n_ratios;
  int32_t n_buckets;
  int32_t l_rule;  // 0 = every stage size 1..L-PP+1, 1 = floor/ceil(L/PP)
};

// ---------------------------------------------------------------------------
// Counting number type.
// ---------------------------------------------------------------------------
uint64_t g_flops = 0;

struct Counted {
  double v;
  Counted() : v(0.0) {}
  Counted(double x) : v(x) {}
};
inline Counted operator+(Counted a, Counted b) { ++g_flops; return Counted(a.v + b.v); }
inline Counted operator-(Counted a, Counted b) { ++g_flops; return Counted(a.v - b.v); }
inline Counted operator*(Counted a, Counted b) { ++g_flops; return Counted(a.v * b.v); }
inline bool operator<(Counted a, Counted b) { return a.v < b.v; }
inline bool operator<=(Counted a, Counted b) { return a.v <= b.v; }
inline bool operator!=(Counted a, Counted b) { return a.v != b.v; }
inline Counted fma3(Counted a, Counted b, Counted c) { g_flops += 2; return Counted(std::fma(a.v, b.v, c.v)); }
inline double val(Counted a) { return a.v; }

inline double fma3(double a, double b, double c) { return std::fma(a, b, c); }
inline double val(double a) { return a; }

template <class R> inline R min2(R a, R b) { return b < a ? b : a; }
template <class R> inline R max2(R a, R b) { return a < b ? b : a; }

// Integer quantities are exact in int64; they enter floating point only below
// 2^53, where the conversion is exact.
inline double exact(int64_t v) {
  const int64_t lim = (int64_t)1 << 53;
  if (v >= lim || v <= -lim) {
    std::fprintf(stderr, "mist oracle: integer %lld is not exactly representable\n", (long long)v);
    std::abort();
  }
  return (double)v;
}

// ---------------------------------------------------------------------------
// Enumeration of the space (Table 2 knobs; groups are the IntraStagePareto
// queries of Eq. 3: hardware sample, G, PP, in-flight count k, layer count l).
// ---------------------------------------------------------------------------
struct Pair { int64_t b, tp, dp; int32_t mb_index; };

struct Group {
  int32_t hw;
  int64_t G, PP, k, l;
  std::vector<Pair> pairs;  // ascending (b, TP)
  uint64_t base;            // id of the group's first configuration
  uint64_t size;            // configurations in the group
};

struct Ctx {
  Model m;
  std::vector<Hw> hw;
  int64_t D, B;
  std::vector<int32_t> mb;
  std::vector<double> r;   // offload ratios
  int32_t R;
  int32_t NB;
  int32_t l_rule;
  std::vector<Group> groups;
  uint64_t n_configs;
  // Host reciprocals, each one correctly rounded division.
  std::vector<double> inv_F, inv_P, inv_L;
  std::vector<std::vector<double>> inv_eta;     // [hw][mb index]
  std::vector<double> psi;                      // [hw][16][4] = 1 / phi
  std::vector<double> om;                       // 1 - r
  std::vector<std::vector<double>> edge;        // [hw][NB]
};

bool valid_model(const Model& m) {
  if (m.arch != 0 && m.arch != 1) return false;
  if (m.n_layers < 1 || m.hidden < 1 || m.heads < 1 || m.kv_heads < 1) return false;
  if (m.ffn < 1 || m.seq < 1 || m.vocab < 1 || m.bytes_w < 1 || m.bytes_opt < 1) return false;
  if (m.hidden % m.heads != 0) return false;
  if (m.heads % m.kv_heads != 0) return false;
  return true;
}

// Tensor-parallel degree TP is admissible when it divides the devices of the
// stage, the attention heads and the MLP width (so every per-rank count is an
// integer), and when KV heads either split evenly or are replicated.
bool tp_ok(const Model& m, int64_t per_stage, int64_t tp) {
  if (per_stage % tp != 0) return false;
  if (m.heads % tp != 0) return false;
  if (m.ffn % tp != 0) return false;
  if (tp <= m.kv_heads) return m.kv_heads % tp == 0;
  return tp % m.kv_heads == 0;
}

bool build_ctx(Ctx& X, const Model* m, const Hw* hw, int32_t n_hw, const Space* s) {
  if (!m || !hw || !s || n_hw < 1) return false;
  if (!valid_model(*m)) return false;
  if (s->n_devices < 1 || s->global_batch < 1 || s->n_mb < 1 || s->n_ratios < 1) return false;
  if (s->n_buckets < 1 || s->n_buckets > 64) return false;
  if (s->l_rule != 0 && s->l_rule != 1) return false;
  X.m = *m;
  X.hw.assign(hw, hw + n_hw);
  X.D = s->n_devices;
  X.B = s->global_batch;
  X.mb.assign(s->mb, s->mb + s->n_mb);
  X.r.assign(s->ratios, s->ratios + s->n_ratios);
  X.R = s->n_ratios;
  X.NB = s->n_buckets;
  X.l_rule = s->l_rule;
  for (size_t i = 0; i < X.mb.size(); ++i) {
    if (X.mb[i] < 1) return false;
    if (i && X.mb[i] <= X.mb[i - 1]) return false;
  }
  for (size_t i = 0; i < X.r.size(); ++i) {
    if (!(X.r[i] >= 0.0 && X.r[i] <= 1.0)) return false;
    if (i && !(X.r[i] > X.r[i - 1])) return false;
  }
  for (const Hw& h : X.hw) {
    if (!(h.flops > 0 && h.mem_bytes > 0 && h.pcie_bw > 0 && h.link_bw > 0)) return false;
    if (!(h.eta_max >= 0 && h.n_half >= 0)) return false;
    if (h.eta_max == 0)
      for (size_t i = 0; i < X.mb.size(); ++i)
        if (!(h.eta_tab[i] > 0 && std::isfinite(h.eta_tab[i]))) return false;
    for (int mask = 0; mask < 16; ++mask)
      for (int j = 0; j < 4; ++j)
        if (!(h.phi[mask][j] >= 1.0 && std::isfinite(h.phi[mask][j]))) return false;
  }

  // Reciprocals and tables.
  X.inv_F.clear(); X.inv_P.clear(); X.inv_L.clear(); X.inv_eta.clear(); X.psi.clear(); X.edge.clear();
  for (const Hw& h : X.hw) {
    X.inv_F.push_back(1.0 / h.flops);
    X.inv_P.push_back(1.0 / h.pcie_bw);
    X.inv_L.push_back(1.0 / h.link_bw);
    std::vector<double> ie;
    for (size_t i = 0; i < X.mb.size(); ++i) {
      if (h.eta_max == 0) {
        // Measured efficiency of this microbatch size; its inverse.
        ie.push_back(1.0 / h.eta_tab[i]);
        continue;
      }
      // Efficiency eta(b) = eta_max * bs / (bs + n_half); its inverse.
      const double bs = exact((int64_t)X.mb[i] * m->seq);
      const double num = bs + h.n_half;
      const double den = h.eta_max * bs;
      ie.push_back(num / den);
    }
    X.inv_eta.push_back(ie);
    for (int mask = 0; mask < 16; ++mask)
      for (int j = 0; j < 4; ++j) X.psi.push_back(1.0 / h.phi[mask][j]);
    std::vector<double> e(X.NB);
    for (int32_t j = 0; j < X.NB; ++j)
      e[j] = (h.mem_bytes * (double)(j + 1)) / (double)X.NB;
    e[X.NB - 1] = h.mem_bytes;
    X.edge.push_back(e);
  }
  X.om.clear();
  for (double v : X.r) X.om.push_back(1.0 - v);

  // Groups, in order hw, PP, G, k, l (all ascending).
  X.groups.clear();
  uint64_t base = 0;
  const int64_t L = m->n_layers;
  for (int32_t ih = 0; ih < n_hw; ++ih) {
    for (int64_t PP = 1; PP <= X.D; ++PP) {
      if (X.D % PP != 0 || PP > L) continue;
      const int64_t per_stage = X.D / PP;
      // Valid (b, TP) pairs and their G = B / (b * DP).
      std::vector<std::pair<int64_t, Pair>> cand;
      for (int32_t bi = 0; bi < (int32_t)X.mb.size(); ++bi) {
        const int64_t b = X.mb[bi];
        for (int64_t tp = 1; tp <= per_stage; ++tp) {
          if (!tp_ok(*m, per_stage, tp)) continue;
          const int64_t dp = per_stage / tp;
          if (X.B % (b * dp) != 0) continue;
          cand.push_back({X.B / (b * dp), Pair{b, tp, dp, bi}});
        }
      }
      std::vector<int64_t> Gs;
      for (auto& c : cand) {
        bool seen = false;
        for (int64_t g : Gs) seen = seen || g == c.first;
        if (!seen) Gs.push_back(c.first);
      }
      for (size_t i = 0; i < Gs.size(); ++i)  // ascending G
        for (size_t j = i + 1; j < Gs.size(); ++j)
          if (Gs[j] < Gs[i]) std::swap(Gs[i], Gs[j]);
      std::vector<int64_t> ls;
      if (X.l_rule == 0) {
        if (PP == 1) ls.push_back(L);
        else for (int64_t l = 1; l <= L - PP + 1; ++l) ls.push_back(l);
      } else {
        const int64_t lo = L / PP, hi = (L + PP - 1) / PP;
        ls.push_back(lo);
        if (hi != lo) ls.push_back(hi);
      }
      for (int64_t G : Gs) {
        std::vector<Pair> ps;
        for (auto& c : cand) if (c.first == G) ps.push_back(c.second);
        for (size_t i = 0; i < ps.size(); ++i)  // ascending (b, TP)
          for (size_t j = i + 1; j < ps.size(); ++j)
            if (ps[j].b < ps[i].b || (ps[j].b == ps[i].b && ps[j].tp < ps[i].tp)) std::swap(ps[i], ps[j]);
        for (int64_t k = 1; k <= PP; ++k) {
          for (int64_t l : ls) {
            Group g;
            g.hw = ih; g.G = G; g.PP = PP; g.k = k; g.l = l; g.pairs = ps;
            g.base = base;
            g.size = (uint64_t)ps.size() * (uint64_t)(l + 1) * 4u *
                     (uint64_t)X.R * X.R * X.R * X.R;
            base += g.size;
            X.groups.push_back(g);
          }
        }
      }
    }
  }
  X.n_configs = base;
  return true;
}

// ---------------------------------------------------------------------------
// Interference model of Sec. 5.2.2 (Algorithm 1) for the four streams
// X = [C (compute), G2G (GPU<->GPU), C2G (host->device), G2C (device->host)],
// written as a simulation of phases.  X[j] is the time stream j needs alone.
// While two or more streams still have work, they all run together and stream
// j progresses phi[set][j] times slower than alone, set being the bit mask of
// the running streams; a phase lasts until the first of them completes.  In a
// phase each member's co-run time is its remaining standalone time times its
// factor, the phase length is the smallest co-run time, and a member's
// standalone time left afterwards is its unused co-run time divided by its
// factor.  The division is a multiplication by the host reciprocal
// psi = 1/phi.  Once at most one stream is left it runs alone; the answer is
// the sum of the phase lengths and that last stream's time.
//
// Each phase ends at least one stream (the shortest co-run time minus itself
// is exactly zero), so there are at most three phases (sets of 4, 3, 2 or
// fewer streams); the loop bound only guards against non-finite input.
// Members are visited in increasing stream index, which fixes the rounding
// order of the minimum and of the final sum.
// ---------------------------------------------------------------------------
inline int popcount4(int v) { return (v & 1) + ((v >> 1) & 1) + ((v >> 2) & 1) + ((v >> 3) & 1); }

template <class R>
R interference(const R Xin[4], const double phi[16][4], const double* psi /*[16][4]*/) {
  R alone[4] = {Xin[0], Xin[1], Xin[2], Xin[3]};  // standalone time still needed per stream
  R elapsed = R(0.0);
  for (int phase = 0; phase < 3; ++phase) {
    int set = 0;
    for (int j = 0; j < 4; ++j)
      if (alone[j] != R(0.0)) set |= 1 << j;
    if (popcount4(set) < 2) break;
    R corun[4];
    R len = R(0.0);
    bool first = true;
    for (int j = 0; j < 4; ++j)
      if (set >> j & 1) {
        corun[j] = alone[j] * R(phi[set][j]);
        len = first ? corun[j] : min2(len, corun[j]);
        first = false;
      }
    for (int j = 0; j < 4; ++j)
      if (set >> j & 1) alone[j] = (corun[j] - len) * R(psi[set * 4 + j]);
    elapsed = elapsed + len;
  }
  for (int j = 0; j < 4; ++j) elapsed = elapsed + alone[j];
  return elapsed;
}

// ---------------------------------------------------------------------------
// Per-configuration cost model, evaluated level by level.
// ---------------------------------------------------------------------------

// Named intermediate terms of one configuration (exposed for the tests).
struct Terms {
  // integers
  int64_t Psi, Pst, Pbuf, atok, afull, ack, Fl, Fh, Xl, Amb, work_c;
  // memory (bytes)
  double S, Wbuf, Gbuf, Obuf, Stash_plus_Off, Rc, Mfwd, Mbwd, Mem;
  // streams (seconds)
  double C, G2Gs, G2Gf, H2Ds, D2Hs, H2Df, D2Hf, ar, r, p2p, H2Dx, D2Hx;
  // results
  double t, T1, d, obj;
};

struct Box { int64_t lo[7], hi[7]; };  // digits: p, c, z, wo, go, oo, ao

// Visitor receives (local id, t, d, mem, obj) and, if non-null, the terms.
template <class R, class Visit>
void walk_group(const Ctx& X, const Group& g, const Box& box, Terms* terms, Visit&& visit) {
  const Model& m = X.m;
  const Hw& hw = X.hw[g.hw];
  const double* psi = &X.psi[(size_t)g.hw * 64];
  const int64_t h = m.hidden, s = m.seq, V = m.vocab, f = m.ffn;
  const int64_t bw = m.bytes_w, bo = m.bytes_opt;
  const bool gpt = m.arch == 0;
  const int64_t l = g.l, PP = g.PP, k = g.k;
  const int64_t Rr = X.R;

  // ---- group level ----
  const int64_t first = (k == PP) ? 1 : 0;   // first stage holds the embedding
  const int64_t last = (k == 1) ? 1 : 0;     // last stage holds the LM head
  const int64_t ke = k < g.G ? k : g.G;      // 1F1B in-flight microbatches
  const R iF = R(X.inv_F[g.hw]), iP = R(X.inv_P[g.hw]), iL = R(X.inv_L[g.hw]);
  const R Gd = R(exact(g.G));

  for (int64_t p = box.lo[0]; p < box.hi[0]; ++p) {
    // ---- pair level: (b, TP, DP) ----
    const Pair& pr = g.pairs[p];
    const int64_t b = pr.b, TP = pr.tp, DP = pr.dp;
    const int64_t dh = h / m.heads;
    const int64_t hkv = (int64_t)m.kv_heads * dh;
    const int64_t hkvr = (TP <= m.kv_heads) ? hkv / TP : dh;  // KV replicated beyond kv_heads
    const int64_t Pq = 2 * h * h;                              // Q and O projections
    const int64_t Pm = (gpt ? 2 : 3) * h * f;                  // MLP (GeLU: 2hf, SwiGLU: 3hf)
    const int64_t Prep = gpt ? 4 * h : 2 * h;                  // two norms, replicated
    const int64_t Psi = (Pq + Pm) / TP + 2 * h * hkvr + Prep;  // per-rank parameters of a layer
    const int64_t Vr = (V + TP - 1) / TP;
    const int64_t Pe = Vr * h + (gpt ? s * h : 0);             // embedding (+ learned positions)
    const int64_t Ph = Vr * h + (gpt ? 2 * h : h);             // LM head + final norm
    const int64_t Pst = l * Psi + first * Pe + last * Ph;      // parameters of the stage
    int64_t Pbuf = Psi;                                        // largest per-layer unit
    if (first * Pe > Pbuf) Pbuf = first * Pe;
    if (last * Ph > Pbuf) Pbuf = last * Ph;
    const int64_t mf = gpt ? 2 : 3;
    // Saved activation elements per token per layer on one rank.
    const int64_t atok = 4 * h + (2 * h + mf * f) / TP + 2 * hkvr + (m.flash ? 0 : (int64_t)m.heads * s / TP);
    const int64_t afull = b * s * bw * atok;                   // bytes, layer not checkpointed
    const int64_t ack = b * s * bw * h;                        // bytes, checkpointed layer input
    // Forward FLOPs per token per layer on one rank (2 per MAC; 4sh attention).
    const int64_t ftok = 2 * ((Pq + Pm) / TP + 2 * h * hkvr) + 4 * s * h / TP;
    const int64_t Fl = b * s * ftok;
    const int64_t Fh = last * 2 * b * s * h * Vr;              // LM head forward FLOPs
    const int64_t Xl = last * 4 * b * s * Vr;                  // fp32 logits (bytes)
    const int64_t p2pB = (int64_t)((k > 1) + (k < PP)) * b * s * h * bw;
    const int64_t arB = 2 * (TP - 1) * (b * s * h * bw / TP);  // ring all-reduce bytes
    const int64_t rB = (DP - 1) * bw * Pst;                    // DP ring step bytes x DP

    const R iD = R(1.0 / exact(DP));
    const R Pw = R(exact(Pst * bw));
    const R Po = R(exact(Pst * bo));
    const R Wb2 = R(exact(2 * Pbuf * bw));
    const R Ob2o = R(exact(2 * Pbuf * bo));
    const R A2 = R(exact(2 * afull));
    const R AF = R(exact(afull));
    const R Xd = R(exact(Xl));
    const R Fld = R(exact(Fl));
    const R Fh3 = R(exact(3 * Fh));
    const R r_ = (R(exact(rB)) * iD) * iL;   // one all-gather or reduce-scatter of the stage
    const R p2p = R(exact(p2pB)) * iL;       // pipeline sends/receives
    const R ar = R(exact(arB)) * iL;         // one TP all-reduce of a (b, s, h) activation
    const R FE = iF * R(X.inv_eta[g.hw][pr.mb_index]);

    for (int64_t c = box.lo[1]; c < box.hi[1]; ++c) {
      // ---- checkpoint level: c recomputed layers ----
      const int64_t Amb = (l - c) * afull + c * ack;  // activations of one microbatch
      const R A = R(exact(Amb));
      const R KA = R(exact(ke * Amb));
      const R Rc = (c > 0) ? AF : R(0.0);             // one recomputed layer's activations
      // Compute stream: fwd + 2x bwd for l layers, one extra forward per
      // recomputed layer, the LM head's fwd + bwd; then the serial TP
      // all-reduces (2 per layer forward, 2 backward, 2 per recomputed layer).
      const R C = fma3(R(exact(4 * l + 2 * c)), ar, fma3(R(exact(3 * l + c)), Fld, Fh3) * FE);

      for (int64_t z = box.lo[2]; z < box.hi[2]; ++z) {
        // ---- ZeRO level ----
        const R sw = (z == 3) ? iD : R(1.0);   // weights sharded
        const R sg = (z >= 2) ? iD : R(1.0);   // gradients sharded
        const R so = (z >= 1) ? iD : R(1.0);   // optimizer states sharded
        const R Sw = Pw * sw;
        const R Sg = Pw * sg;
        const R So = Po * so;
        const R HWz = R(2.0) * Sw;             // weights fetched for fwd and bwd
        static const double ms_tab[4] = {0.0, 0.0, 1.0, 3.0};  // per microbatch: z2 RS; z3 AG+AG+RS
        static const double mf_tab[4] = {2.0, 2.0, 2.0, 3.0};  // first: + AR (z0), RS+AG (z1), AG (z2)
        const R G2Gs = fma3(R(ms_tab[z]), r_, p2p);
        const R G2Gf = fma3(R(mf_tab[z]), r_, p2p);
        const R Obo = Ob2o * so;
        const R Obg = Wb2 * sg;

        for (int64_t iw = box.lo[3]; iw < box.hi[3]; ++iw) {
          // ---- weight offload level ----
          const R rw = R(X.r[iw]), qw = R(X.om[iw]);
          const R Sww = qw * Sw;                          // resident weights
          const R Wbuf = Wb2 * (R(1.0) - qw * sw);        // double-buffered fetched weights
          const R HW = rw * HWz;
          const R DW = rw * Sw;                           // updated weights written back

          for (int64_t ig = box.lo[4]; ig < box.hi[4]; ++ig) {
            // ---- gradient offload level ----
            const R rg = R(X.r[ig]), qg = R(X.om[ig]);
            const R Swg = fma3(qg, Sg, Sww);
            const R Gbuf = Wb2 * (R(1.0) - qg * sg);      // double-buffered gradient unit
            const R DG = rg * Sg;                         // offloaded gradient bytes
            const R Og = rg * Obg;

            for (int64_t io = box.lo[5]; io < box.hi[5]; ++io) {
              // ---- optimizer-state offload level ----
              const R ro = R(X.r[io]), qo = R(X.om[io]);
              const R S = fma3(qo, So, Swg);              // resident model states
              const R Obuf = fma3(ro, Obo, Og);           // optimizer-step working unit
              const R HX = fma3(ro, So, DG);              // fetched before the first forward
              const R DX = fma3(ro, So, DW);              // written back after the step
              const R base = S + Wbuf;
              const R BF = (base + Obuf) + Xd;
              const R BB = ((base + Gbuf) + Rc) + Xd;
              const R H2Dx = HX * iP;
              const R D2Hx = DX * iP;

              for (int64_t ia = box.lo[6]; ia < box.hi[6]; ++ia) {
                // ---- activation offload level: one configuration ----
                const R ra = R(X.r[ia]), qa = R(X.om[ia]);
                const R SO = fma3(ra, A2, qa * KA);       // stashed + double-buffered offload
                const R Mf = BF + SO;
                const R Mb = BB + SO;
                const R Mem = max2(Mf, Mb);
                const R H2Ds = fma3(ra, A, HW) * iP;
                const R D2Hs = fma3(ra, A, DG) * iP;
                const R H2Df = H2Ds + H2Dx;
                const R D2Hf = D2Hs + D2Hx;
                const R Xs[4] = {C, G2Gs, H2Ds, D2Hs};
                const R Xf[4] = {C, G2Gf, H2Df, D2Hf};
                const R t = interference(Xs, hw.phi, psi);
                const R T1 = interference(Xf, hw.phi, psi);
                const R d = T1 - t;
                const R obj = fma3(Gd, t, d);

                const int64_t local =
                    ((((((p * (l + 1) + c) * 4 + z) * Rr + iw) * Rr + ig) * Rr + io) * Rr + ia);
                if (terms) {
                  Terms& T = *terms;
                  T.Psi = Psi; T.Pst = Pst; T.Pbuf = Pbuf; T.atok = atok; T.afull = afull; T.ack = ack;
                  T.Fl = Fl; T.Fh = Fh; T.Xl = Xl; T.Amb = Amb; T.work_c = (3 * l + c) * Fl + 3 * Fh;
                  T.S = val(S); T.Wbuf = val(Wbuf); T.Gbuf = val(Gbuf); T.Obuf = val(Obuf);
                  T.Stash_plus_Off = val(SO); T.Rc = val(Rc); T.Mfwd = val(Mf); T.Mbwd = val(Mb);
                  T.Mem = val(Mem); T.C = val(C); T.G2Gs = val(G2Gs); T.G2Gf = val(G2Gf);
                  T.H2Ds = val(H2Ds); T.D2Hs = val(D2Hs); T.H2Df = val(H2Df); T.D2Hf = val(D2Hf);
                  T.ar = val(ar); T.r = val(r_); T.p2p = val(p2p); T.H2Dx = val(H2Dx); T.D2Hx = val(D2Hx);
                  T.t = val(t); T.T1 = val(T1); T.d = val(d); T.obj = val(obj);
                }
                visit(local, val(t), val(d), val(Mem), val(obj));
              }
            }
          }
        }
      }
    }
  }
}

Box full_box(const Ctx& X, const Group& g) {
  Box b;
  const int64_t hi[7] = {(int64_t)g.pairs.size(), g.l + 1, 4, X.R, X.R, X.R, X.R};
  for (int i = 0; i < 7; ++i) { b.lo[i] = 0; b.hi[i] = hi[i]; }
  return b;
}

// Splits a local id into its digits (innermost first: ao, oo, go, wo, z, c, p).
Box single_box(const Ctx& X, const Group& g, uint64_t local) {
  const int64_t R = X.R;
  int64_t dig[7];
  uint64_t v = local;
  dig[6] = (int64_t)(v % R); v /= R;
  dig[5] = (int64_t)(v % R); v /= R;
  dig[4] = (int64_t)(v % R); v /= R;
  dig[3] = (int64_t)(v % R); v /= R;
  dig[2] = (int64_t)(v % 4); v /= 4;
  dig[1] = (int64_t)(v % (uint64_t)(g.l + 1)); v /= (uint64_t)(g.l + 1);
  dig[0] = (int64_t)v;
  Box b;
  for (int i = 0; i < 7; ++i) { b.lo[i] = dig[i]; b.hi[i] = dig[i] + 1; }
  return b;
}

int find_group(const Ctx& X, uint64_t id) {
  if (id >= X.n_configs) return -1;
  size_t lo = 0, hi = X.groups.size();  // last group with base <= id
  while (hi - lo > 1) {
    const size_t mid = (lo + hi) / 2;
    if (X.groups[mid].base <= id) lo = mid; else hi = mid;
  }
  return (int)lo;
}

int32_t bucket_of(const Ctx& X, int32_t hw, double mem) {
  for (int32_t j = 0; j < X.NB; ++j)
    if (mem <= X.edge[hw][j]) return j;
  return -1;  // infeasible
}

// (obj, id) lexicographic order.
inline bool lex_less(double o1, uint64_t i1, double o2, uint64_t i2) {
  return o1 < o2 || (o1 == o2 && i1 < i2);
}

void check_values(double t, double d, double mem, double obj) {
  if (!(std::isfinite(t) && std::isfinite(d) && std::isfinite(mem) && std::isfinite(obj)) ||
      !(t > 0.0) || !(mem > 0.0) || !(obj > 0.0) || std::signbit(d) != (d < 0.0)) {
    std::fprintf(stderr, "mist oracle: non-finite, non-positive or negative-zero value\n");
    std::abort();
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// C entry points (ctypes).
// ---------------------------------------------------------------------------
extern "C" {

struct orc_group_key {
  int32_t hw, n_pairs;
  int64_t G, PP, k, l;
  uint64_t base, size;
};

struct orc_terms {
  int64_t Psi, Pst, Pbuf, atok, afull, ack, Fl, Fh, Xl, Amb, work_c;
  double S, Wbuf, Gbuf, Obuf, Stash_plus_Off, Rc, Mfwd, Mbwd, Mem;
  double C, G2Gs, G2Gf, H2Ds, D2Hs, H2Df, D2Hf, ar, r, p2p, H2Dx, D2Hx;
  double t, T1, d, obj;
};
static_assert(sizeof(orc_terms) == sizeof(Terms), "terms layout");

int orc_space_info(const Model* m, const Hw* hw, int32_t n_hw, const Space* s,
                   uint64_t* n_configs, int64_t* n_groups) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  *n_configs = X.n_configs;
  *n_groups = (int64_t)X.groups.size();
  return 0;
}

int orc_group_keys(const Model* m, const Hw* hw, int32_t n_hw, const Space* s,
                   int64_t g0, int64_t n, orc_group_key* out) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g0 < 0 || n < 0 || g0 + n > (int64_t)X.groups.size()) return -5;
  for (int64_t i = 0; i < n; ++i) {
    const Group& g = X.groups[g0 + i];
    out[i].hw = g.hw; out[i].n_pairs = (int32_t)g.pairs.size();
    out[i].G = g.G; out[i].PP = g.PP; out[i].k = g.k; out[i].l = g.l;
    out[i].base = g.base; out[i].size = g.size;
  }
  return 0;
}

// Decodes an id into (hw, G, PP, k, l, b, TP, DP, z, c, wo, go, oo, ao digit indices).
int orc_decode(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, uint64_t id, int64_t* out14) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  const int gi = find_group(X, id);
  if (gi < 0) return -5;
  const Group& g = X.groups[gi];
  const Box b = single_box(X, g, id - g.base);
  const Pair& p = g.pairs[b.lo[0]];
  const int64_t v[14] = {g.hw, g.G, g.PP, g.k, g.l, p.b, p.tp, p.dp,
                         b.lo[2], b.lo[1], b.lo[3], b.lo[4], b.lo[5], b.lo[6]};
  for (int i = 0; i < 14; ++i) out14[i] = v[i];
  return 0;
}

// Per-configuration values for arbitrary ids: out[4*i..] = t, d, mem, obj.
int orc_eval_ids(const Model* m, const Hw* hw, int32_t n_hw, const Space* s,
                 const uint64_t* ids, int64_t n, double* out) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  for (int64_t i = 0; i < n; ++i) {
    const int gi = find_group(X, ids[i]);
    if (gi < 0) return -5;
    const Group& g = X.groups[gi];
    const Box b = single_box(X, g, ids[i] - g.base);
    walk_group<double>(X, g, b, nullptr, [&](int64_t, double t, double d, double mem, double obj) {
      out[4 * i + 0] = t; out[4 * i + 1] = d; out[4 * i + 2] = mem; out[4 * i + 3] = obj;
    });
  }
  return 0;
}

int orc_eval_terms(const Model* m, const Hw* hw, int32_t n_hw, const Space* s,
                   uint64_t id, orc_terms* out) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  const int gi = find_group(X, id);
  if (gi < 0) return -5;
  const Group& g = X.groups[gi];
  Terms T;
  walk_group<double>(X, g, single_box(X, g, id - g.base), &T, [](int64_t, double, double, double, double) {});
  std::memcpy(out, &T, sizeof(T));
  return 0;
}

// Algorithm 1 alone, for the tests: phi[16][4] factors, X[4] stream times.
double orc_interference(const double* X4, const double* phi64) {
  double phi[16][4];
  double psi[64];
  for (int i = 0; i < 64; ++i) {
    phi[i / 4][i % 4] = phi64[i];
    psi[i] = 1.0 / phi64[i];
  }
  const double X[4] = {X4[0], X4[1], X4[2], X4[3]};
  return interference<double>(X, phi, psi);
}

// FP64 operations of Algorithm 1 alone on one stream vector (the counting build of the
// same template), for the tests that pin the counter by hand.
int orc_count_interference(const double* X4, const double* phi64, uint64_t* flops) {
  double phi[16][4];
  double psi[64];
  for (int i = 0; i < 64; ++i) {
    phi[i / 4][i % 4] = phi64[i];
    psi[i] = 1.0 / phi64[i];
  }
  const Counted X[4] = {Counted(X4[0]), Counted(X4[1]), Counted(X4[2]), Counted(X4[3])};
  g_flops = 0;
  (void)interference<Counted>(X, phi, psi);
  *flops = g_flops;
  return 0;
}

// Every configuration of groups [g0, g1): out[5*i..] = t, d, mem, obj, bucket
// (bucket -1 = infeasible), in id order starting at groups[g0].base.
int orc_dump(const Model* m, const Hw* hw, int32_t n_hw, const Space* s,
             int64_t g0, int64_t g1, double* out, uint64_t cap) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g0 < 0 || g1 < g0 || g1 > (int64_t)X.groups.size()) return -5;
  uint64_t need = 0;
  for (int64_t gi = g0; gi < g1; ++gi) need += X.groups[gi].size;
  if (need > cap) return -5;
  uint64_t w = 0;
  for (int64_t gi = g0; gi < g1; ++gi) {
    const Group& g = X.groups[gi];
    walk_group<double>(X, g, full_box(X, g), nullptr, [&](int64_t, double t, double d, double mem, double obj) {
      out[5 * w + 0] = t; out[5 * w + 1] = d; out[5 * w + 2] = mem; out[5 * w + 3] = obj;
      out[5 * w + 4] = (double)bucket_of(X, g.hw, mem);
      ++w;
    });
  }
  return 0;
}

// The tuner's reductions for groups [g0, g1):
//   bucket_best: per group, per bucket j < NB, the (obj, id) lexicographic
//                minimum over feasible configurations whose bucket is j
//                (id = UINT64_MAX, obj = +inf when the bucket is empty);
//   best:        per group, the lexicographic minimum over all feasible ones;
//   frontier:    bit j set when bucket j is non-empty and its obj is strictly
//                below every obj of a lower bucket.
int orc_run(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, int64_t g0, int64_t g1,
            uint64_t* best_id, double* best_obj, uint64_t* bucket_id, double* bucket_obj,
            uint64_t* frontier) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g0 < 0 || g1 < g0 || g1 > (int64_t)X.groups.size()) return -5;
  const double inf = std::numeric_limits<double>::infinity();
  const uint64_t none = UINT64_MAX;
  for (int64_t gi = g0; gi < g1; ++gi) {
    const Group& g = X.groups[gi];
    const int64_t o = gi - g0;
    std::vector<uint64_t> bid(X.NB, none);
    std::vector<double> bobj(X.NB, inf);
    walk_group<double>(X, g, full_box(X, g), nullptr, [&](int64_t local, double t, double d, double mem, double obj) {
      check_values(t, d, mem, obj);
      const int32_t j = bucket_of(X, g.hw, mem);   // Eq. 4 constraint: mem <= budget
      if (j < 0) return;
      const uint64_t id = g.base + (uint64_t)local;
      if (lex_less(obj, id, bobj[j], bid[j])) { bobj[j] = obj; bid[j] = id; }
    });
    uint64_t bi = none;
    double bo = inf;
    uint64_t mask = 0;
    double below = inf;
    for (int32_t j = 0; j < X.NB; ++j) {
      bucket_id[o * X.NB + j] = bid[j];
      bucket_obj[o * X.NB + j] = bobj[j];
      if (bid[j] == none) continue;
      if (lex_less(bobj[j], bid[j], bo, bi)) { bo = bobj[j]; bi = bid[j]; }
      if (bobj[j] < below) mask |= (uint64_t)1 << j;
      below = min2(below, bobj[j]);
    }
    best_id[o] = bi;
    best_obj[o] = bo;
    frontier[o] = mask;
  }
  return 0;
}

// Eq. 4 with sampled weights (Sec. 5.3): for each sample alpha_a, the feasible
// configuration of the group that minimises alpha_a * G * t + (1 - alpha_a) * d, the
// lowest id among equal values.  The value is fma(alpha_a * G, t, (1 - alpha_a) * d), with
// alpha_a * G (per group) and 1 - alpha_a (per sample) each rounded once.  A group with no
// feasible configuration gets UINT64_MAX and +inf.  Outputs are [g1 - g0][n_alpha].
int orc_run_alpha(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, const double* alphas,
                  int32_t n_alpha, int64_t g0, int64_t g1, uint64_t* out_id, double* out_obj) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g0 < 0 || g1 < g0 || g1 > (int64_t)X.groups.size()) return -5;
  if (n_alpha < 1 || n_alpha > 16) return -1;
  for (int32_t a = 0; a < n_alpha; ++a)
    if (!(alphas[a] >= 0.0 && alphas[a] <= 1.0)) return -1;
  const double inf = std::numeric_limits<double>::infinity();
  std::vector<double> beta(n_alpha), aG(n_alpha);
  for (int32_t a = 0; a < n_alpha; ++a) beta[a] = 1.0 - alphas[a];
  for (int64_t gi = g0; gi < g1; ++gi) {
    const Group& g = X.groups[gi];
    const int64_t o = gi - g0;
    for (int32_t a = 0; a < n_alpha; ++a) {
      aG[a] = alphas[a] * exact(g.G);
      out_id[o * n_alpha + a] = UINT64_MAX;
      out_obj[o * n_alpha + a] = inf;
    }
    walk_group<double>(X, g, full_box(X, g), nullptr, [&](int64_t local, double t, double d, double mem, double obj) {
      check_values(t, d, mem, obj);
      if (bucket_of(X, g.hw, mem) < 0) return;  // Eq. 4 constraint: mem <= budget
      const uint64_t id = g.base + (uint64_t)local;
      for (int32_t a = 0; a < n_alpha; ++a) {
        const double v = std::fma(aG[a], t, beta[a] * d);
        if (lex_less(v, id, out_obj[o * n_alpha + a], out_id[o * n_alpha + a])) {
          out_obj[o * n_alpha + a] = v;
          out_id[o * n_alpha + a] = id;
        }
      }
    });
  }
  return 0;
}

// Exact time-vs-memory frontier of group g (the staircase without memory buckets): the
// feasible configurations ordered by (mem, obj, id); one is on the frontier when its obj is
// strictly below the obj of every configuration before it.  Writes up to cap points in that
// order (increasing mem, strictly decreasing obj) and the count to *n_out; returns -5 when
// cap is too small (with *n_out set to the count).
int orc_pareto_exact(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, int64_t g_index,
                     uint64_t* out_id, double* out_obj, double* out_mem, int64_t cap, int64_t* n_out) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g_index < 0 || g_index >= (int64_t)X.groups.size()) return -5;
  const Group& g = X.groups[g_index];
  struct P { double mem, obj; uint64_t id; };
  std::vector<P> all;
  walk_group<double>(X, g, full_box(X, g), nullptr, [&](int64_t local, double t, double d, double mem, double obj) {
    check_values(t, d, mem, obj);
    if (bucket_of(X, g.hw, mem) < 0) return;  // Eq. 4 constraint: mem <= budget
    all.push_back(P{mem, obj, g.base + (uint64_t)local});
  });
  std::sort(all.begin(), all.end(), [](const P& a, const P& b) {
    if (a.mem != b.mem) return a.mem < b.mem;
    if (a.obj != b.obj) return a.obj < b.obj;
    return a.id < b.id;
  });
  int64_t n = 0;
  double run = std::numeric_limits<double>::infinity();
  for (const P& p : all) {
    if (p.obj < run) {
      if (n < cap) { out_id[n] = p.id; out_obj[n] = p.obj; out_mem[n] = p.mem; }
      ++n;
    }
    run = min2(run, p.obj);
  }
  *n_out = n;
  return n > cap ? -5 : 0;
}

// FP64 operations of the definition over groups [g0, g1), counted by running
// the same templates on the counting type.
int orc_count_flops(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, int64_t g0, int64_t g1,
                    uint64_t* flops, uint64_t* configs) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  if (g0 < 0 || g1 < g0 || g1 > (int64_t)X.groups.size()) return -5;
  g_flops = 0;
  uint64_t n = 0;
  for (int64_t gi = g0; gi < g1; ++gi) {
    const Group& g = X.groups[gi];
    walk_group<Counted>(X, g, full_box(X, g), nullptr, [&](int64_t, double, double, double, double) { ++n; });
  }
  *flops = g_flops;
  *configs = n;
  return 0;
}

// FP64 operations of the definition for single configurations evaluated from scratch: every
// level of ids[i] once, nothing shared with other configurations.
int orc_count_flops_ids(const Model* m, const Hw* hw, int32_t n_hw, const Space* s, const uint64_t* ids,
                        int64_t n, uint64_t* flops) {
  Ctx X;
  if (!build_ctx(X, m, hw, n_hw, s)) return -1;
  g_flops = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int gi = find_group(X, ids[i]);
    if (gi < 0) return -5;
    const Group& g = X.groups[gi];
    walk_group<Counted>(X, g, single_box(X, g, ids[i] - g.base), nullptr, [](int64_t, double, double, double, double) {});
  }
  *flops = g_flops;
  return 0;
}

}  // extern "C"
