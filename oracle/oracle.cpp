// CPU oracle for the PackServe window scorer.  TEST INFRASTRUCTURE ONLY:
// only the tests, the smoke check and the benchmark's CPU-baseline leg may
// load or call it.  The GPU library never links, includes or calls it, and
// it shares no code, header, table or constant generator with that library.
//
// It is the plain, slow, obviously correct reading of the paper's method:
// Algorithm 1 (KVC-first, SLO-aware request packing) taken step by step for
// one request at a time, in fp64 (fp32 interface values are widened
// exactly), with a naive block-by-block prefix walk over a hash set per
// instance and an exhaustive selection over all instances.
//
// Functions and what pins them (tests under tests/ marked "not gpu"):
//   prefix_hit      - longest cached prefix (Sec. 7, local prefix tree; the
//                     N new / C cached split of Sec. 5.2).  Pinned by brute-
//                     force token-level longest-common-prefix on tiny windows
//                     and by the generator's construction (owner hits).
//   t_prefill       - Eq. 7 plus the empirical C and C^2 terms of Sec. 5.3.
//                     Pinned by hand-computed cases and special cases.
//   recompute_cost, cache_benefit, filter - Eq. 9 with Alg. 1's KVC-first
//                     stage.  Pinned by the hand-worked example and the
//                     eta = 0 / Z = 0 special cases the paper states.
//   predict_tpot    - Eq. 10 with the per-segment decode model of Eq. 8 and
//                     the EMA factor of Sec. 5.3.  Pinned by hand cases, the
//                     A = 0 special case and the single-segment reduction.
//   select          - decode-batch-size-centric key (Sec. 6.2, Table 4's
//                     D-C-Q) and the cache-aware load-balancing fallback
//                     (LMetric product, Sec. 8.1 baselines).  Pinned by hand
//                     cases, exhaustive brute force and invariants.
//   commit          - sequential application of decisions (Sec. 7: state is
//                     updated along the request path).  Pinned by a
//                     hand-traced sequence.
//   schedule        - Algorithm 1 per arrival: score, then commit, request
//                     by request.  Pinned by the round-robin closed form on
//                     identical instances, capacity exhaustion, a hand-traced
//                     session that follows its own blocks, and the TPOT
//                     guarantee of every placement at its arrival.
//   replay          - latencies of given placements at their arrival, then
//                     commit.  Pinned by a hand-traced sequence.
//
// parity unpinned (the paper leaves these open; the oracle follows the
// readings listed in the design notes and only hand cases of those readings
// pin it): the capacity rule behind CapacityCandidates (A_i + 1 <= B_max and
// S_i + L_r <= M_KV), the projected context S+ = S_i + L_r, the queueing
// estimate alpha0 * Q_i + alpha1 * P_i inside predicted TTFT, snapshot
// semantics within a window, and the outputs of a rejected request.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <unordered_set>
#include <vector>

#include <omp.h>

extern "C" {

// Oracle-local model/policy description (fp64).  The Python wrapper widens
// the fp32 interface coefficients into it exactly.
typedef struct {
  double alpha[6];      // T_pf(N, C) = a0 + a1 N + a2 N C + a3 N^2 + a4 C + a5 C^2
  int32_t n_seg;        // decode segments
  int32_t seg_ub[32];   // inclusive upper batch size of each segment, ascending
  double beta[32][3];   // T_iter(B, S) = b0 + b1 B + b2 S, per segment
  double gamma[32];     // EMA factor per segment
  double eta;           // recomputation budget
  double tau;           // TPOT target
  double ttft_floor;    // minimum TTFT budget
  double lout;          // recent median output length
  int32_t block_tokens; // tokens per block
  int32_t b_max;        // engine batch limit
  int64_t kv_cap;       // KV capacity, tokens
  uint32_t flags;       // 1 TTFT admission, 2 no KVC filter, 4 no TPOT filter,
                        // 8 fallback by the D-C-Q key; bits 8..11 selector
  uint64_t rand_seed;   // seed of the random selector's stream
} orc_model;

}  // extern "C"

namespace {

constexpr uint32_t F_TTFT_ADMIT = 1u, F_NO_KVC = 2u, F_NO_TPOT = 4u, F_FALLBACK_DCQ = 8u;
// Selection orders within T (Table 4 of the paper, plus LMetric alone).
enum Selector : uint32_t { SEL_DCQ = 0, SEL_D, SEL_DQ, SEL_DC, SEL_DQC, SEL_HCQ, SEL_RANDOM, SEL_LMETRIC };
constexpr uint32_t R_REJECT = 1u, R_FALLBACK = 2u, R_TTFT_MISS = 4u;
// Near-boundary bits.  NB_RHO, NB_TPOT, NB_TTFT, NB_Z and NB_HEADROOM mark a
// decision (instance, hit, flags) that rounding may change; NB_MISSFLAG marks
// a TTFT_MISS flag that rounding may change; NB_SIZES marks a |T| that
// rounding may change while the decision cannot.  Bits 16..31 count the
// candidates behind NB_SIZES.
constexpr uint32_t NB_RHO = 1u, NB_TPOT = 2u, NB_TTFT = 4u, NB_Z = 8u, NB_MISSFLAG = 16u,
                   NB_HEADROOM = 32u, NB_SIZES = 64u;
constexpr double NB_REL = 1e-5;

struct Snapshot {
  int32_t n_inst = 0;
  int32_t cap = 0;
  std::vector<int32_t> out_lens;  // every recorded output length, in order
  std::vector<std::unordered_set<uint64_t>> sets;
  std::vector<int32_t> D, Q;
  std::vector<int64_t> P, S;
};

struct Chain {
  const uint64_t* a;
  int32_t na;
  const uint64_t* b;
  int32_t nb;
  int32_t len() const { return na + nb; }
  uint64_t at(int32_t j) const { return j < na ? a[j] : b[j - na]; }
};

// Longest cached prefix, in blocks: walk the chain from its first block and
// stop at the first block the instance does not hold.
int64_t prefix_hit(const std::unordered_set<uint64_t>& set, const Chain& ch) {
  int32_t j = 0;
  while (j < ch.len() && set.count(ch.at(j)) != 0) ++j;
  return j;
}

// Eq. 7 with the two empirical cache terms: N new tokens, C cached tokens.
double t_prefill(const orc_model& m, double N, double C) {
  const double* a = m.alpha;
  return a[0] + a[1] * N + a[2] * N * C + a[3] * N * N + a[4] * C + a[5] * C * C;
}

// Decode segment for a projected batch size: the first segment whose
// inclusive upper bound covers it, else the last one.
int segment_of(const orc_model& m, int64_t B) {
  for (int s = 0; s < m.n_seg; ++s)
    if (B <= m.seg_ub[s]) return s;
  return m.n_seg - 1;
}

// Eq. 10's TPOT and Eq. 4's TTFT of placing a request of L tokens (n new,
// c cached) on instance i in the current state: the decode step of the
// projected batch and context scaled by its segment's factor, plus the
// request's prefill amortised over the median output length when the
// instance is busy; the prefill plus the queueing estimate.
void candidate_latency(const Snapshot& sn, const orc_model& m, int32_t i, int64_t n, int64_t c,
                       int64_t L, double& tpot, double& ttft) {
  const int64_t active = (int64_t)sn.D[i] + sn.Q[i];
  const int64_t Bp = active + 1;
  const double Sp = (double)(sn.S[i] + L);
  const int s = segment_of(m, Bp);
  const double t_iter = m.gamma[s] * (m.beta[s][0] + m.beta[s][1] * (double)Bp + m.beta[s][2] * Sp);
  const double tpf = t_prefill(m, (double)n, (double)c);
  const double interference = active > 0 ? tpf / std::max(1.0, m.lout) : 0.0;
  tpot = t_iter + interference;
  ttft = tpf + m.alpha[0] * (double)sn.Q[i] + m.alpha[1] * (double)sn.P[i];
}

struct Cand {
  int32_t i;
  int64_t hit;  // blocks
  int64_t n, c; // new / cached tokens
  double W;     // recomputation cost
  double rho;
  double tpot, ttft;
  bool inC, inT;
  bool unsure;  // member of C whose T membership rounding may change
};

struct Decision {
  int32_t inst;
  int32_t hit;
  double ttft, tpot;
  uint32_t flags;
  uint32_t nA, nC, nT;
  uint32_t nb;
};

// Algorithm 1 for one request against the snapshot.  Fills every
// capacity-eligible candidate (with its memberships) into A and returns the
// decision.
// SplitMix64 (Steele, Lea, Flood; Vigna's reference): the (r + 1)-th output
// of the stream seeded with `seed`.
uint64_t rand_seed_state(uint64_t seed, int64_t r) {
  uint64_t z = seed + (uint64_t)(r + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

Decision score_one(const Snapshot& sn, const orc_model& m, const Chain& ch, std::vector<Cand>& A,
                   int64_t r_index) {
  Decision d{-1, 0, 0.0, 0.0, R_REJECT, 0, 0, 0, 0};
  const int64_t L = (int64_t)ch.len() * m.block_tokens;
  const double Ld = (double)L;

  // Capacity guard: instances that can take one more active request and the
  // request's tokens.
  A.clear();
  for (int32_t i = 0; i < sn.n_inst; ++i) {
    int64_t active = (int64_t)sn.D[i] + sn.Q[i];
    if (active + 1 <= m.b_max && sn.S[i] + L <= m.kv_cap) {
      Cand c{};
      c.i = i;
      A.push_back(c);
    }
  }
  d.nA = (uint32_t)A.size();
  if (A.empty()) return d;

  // KVC-first recomputation filtering.
  const double tpf_cached = t_prefill(m, 0.0, Ld);  // fully cached input
  const double tpf_cold = t_prefill(m, Ld, 0.0);    // fully uncached input
  double Wmin = INFINITY;
  int64_t hit_at_min = -1;  // hit of the first minimiser (for the near-boundary rule)
  for (Cand& c : A) {
    c.hit = prefix_hit(sn.sets[c.i], ch);
    c.c = c.hit * m.block_tokens;
    c.n = L - c.c;
    c.W = std::max(0.0, t_prefill(m, (double)c.n, (double)c.c) - tpf_cached);
    if (c.W < Wmin) {
      Wmin = c.W;
      hit_at_min = c.hit;
    }
  }
  const double Z = tpf_cold - tpf_cached;
  const bool kvc_on = !(m.flags & F_NO_KVC);
  // A fully cached candidate has W = 0 exactly, so W_min = 0 exactly; a
  // candidate with nothing cached has W = Z (the same expression), so its
  // rho is then exactly 1 under any rounding.
  bool some_full = false;
  for (const Cand& c : A) some_full |= c.n == 0;
  if (kvc_on && std::fabs(Z) <= NB_REL * std::fabs(tpf_cold)) d.nb |= NB_Z;
  for (Cand& c : A) {
    if (!kvc_on || Z <= 0.0) {
      c.rho = 0.0;
      c.inC = true;
    } else {
      c.rho = (c.W - Wmin) / Z;
      c.inC = c.rho <= m.eta;
      // A candidate with the minimiser's own hit has rho = 0 exactly under
      // any rounding, and so has one with nothing cached rho = 1 when the
      // minimiser is fully cached; every other rho within the relative
      // window of eta is decided by rounding.
      const bool exact_zero = c.W == Wmin && c.hit == hit_at_min;
      const bool exact_one = some_full && c.c == 0;
      if (!exact_zero && !exact_one && std::fabs(c.rho - m.eta) <= NB_REL * std::max(m.eta, 1.0))
        d.nb |= NB_RHO;
    }
  }

  // SLO-aware admission (Eq. 10) and the TTFT estimate (Eq. 4).
  const double slo = std::max(m.ttft_floor, tpf_cold);
  // A candidate with nothing cached and nothing queued has TTFT = T_pf(L, 0),
  // the very quantity the budget is (when it exceeds the floor): the two are
  // equal in any precision, so that comparison is never near a boundary.
  auto ttft_is_budget = [&](const Cand& c) {
    return c.c == 0 && sn.Q[c.i] == 0 && sn.P[c.i] == 0 && tpf_cold >= m.ttft_floor;
  };
  for (Cand& c : A) {
    candidate_latency(sn, m, c.i, c.n, c.c, L, c.tpot, c.ttft);
    const bool tpot_ok = (m.flags & F_NO_TPOT) || c.tpot < m.tau;
    const bool ttft_ok = !(m.flags & F_TTFT_ADMIT) || c.ttft <= slo;
    c.inT = c.inC && tpot_ok && ttft_ok;
    // T membership is decided by rounding when a test it needs lies within
    // the relative window of its bound and the other test passes or is
    // itself that close.
    const bool tpot_near = !(m.flags & F_NO_TPOT) && std::fabs(c.tpot - m.tau) <= NB_REL * m.tau;
    const bool ttft_near = (m.flags & F_TTFT_ADMIT) && !ttft_is_budget(c) &&
                           std::fabs(c.ttft - slo) <= NB_REL * slo;
    c.unsure = c.inC && ((tpot_near && (ttft_ok || ttft_near)) || (ttft_near && (tpot_ok || tpot_near)));
    if (c.unsure) d.nb |= NB_SIZES;
  }
  uint32_t n_unsure = 0;
  for (const Cand& c : A) {
    d.nC += c.inC;
    d.nT += c.inT;
    n_unsure += c.unsure;
  }
  // bits 16..31: how many candidates' T membership rounding may change
  // (|T| can differ by at most that many), saturated
  d.nb |= std::min<uint32_t>(n_unsure, 0xFFFFu) << 16;

  // Packing within T by the selector; D-C-Q by default (most decoding
  // requests, then most cached blocks, then fewest queued, then lowest id).
  const uint32_t sel = (m.flags >> 8) & 0xFu;
  auto lmetric = [&](const Cand& c) {
    const int64_t active = (int64_t)sn.D[c.i] + sn.Q[c.i];
    return (unsigned __int128)(uint64_t)(sn.P[c.i] + c.n) * (unsigned __int128)(uint64_t)(active + 1);
  };
  // true if a comes before b in selector order s
  auto before = [&](uint32_t s, const Cand& a, const Cand& b) {
    const int32_t Da = sn.D[a.i], Db = sn.D[b.i], Qa = sn.Q[a.i], Qb = sn.Q[b.i];
    switch (s) {
      case SEL_D:
        if (Da != Db) return Da > Db;
        break;
      case SEL_DQ:
        if (Da != Db) return Da > Db;
        if (Qa != Qb) return Qa < Qb;
        break;
      case SEL_DC:
        if (Da != Db) return Da > Db;
        if (a.hit != b.hit) return a.hit > b.hit;
        break;
      case SEL_DQC:
        if (Da != Db) return Da > Db;
        if (Qa != Qb) return Qa < Qb;
        if (a.hit != b.hit) return a.hit > b.hit;
        break;
      case SEL_HCQ: {  // smallest TPOT headroom first
        const double ha = m.tau - a.tpot, hb = m.tau - b.tpot;
        if (ha != hb) return ha < hb;
        if (a.hit != b.hit) return a.hit > b.hit;
        if (Qa != Qb) return Qa < Qb;
        break;
      }
      case SEL_LMETRIC: {
        const unsigned __int128 la = lmetric(a), lb = lmetric(b);
        if (la != lb) return la < lb;
        break;
      }
      default:  // SEL_DCQ
        if (Da != Db) return Da > Db;
        if (a.hit != b.hit) return a.hit > b.hit;
        if (Qa != Qb) return Qa < Qb;
        break;
    }
    return a.i < b.i;
  };
  const Cand* best = nullptr;
  if (sel == SEL_RANDOM) {
    // The k-th member of T in id order, k from the (r + 1)-th output of a
    // SplitMix64 stream seeded with rand_seed: k = floor(z_hi * |T| / 2^32).
    if (d.nT > 0) {
      uint64_t z = rand_seed_state(m.rand_seed, r_index);
      const uint64_t k = ((z >> 32) * (uint64_t)d.nT) >> 32;
      uint64_t seen = 0;
      for (const Cand& c : A) {
        if (!c.inT) continue;
        if (seen++ == k) {
          best = &c;
          break;
        }
      }
    }
  } else {
    for (const Cand& c : A) {
      if (c.inT && (!best || before(sel, c, *best))) best = &c;
    }
    if (sel == SEL_HCQ && best) {
      const double hb = m.tau - best->tpot;
      for (const Cand& c : A)
        if (c.inT && &c != best && std::fabs((m.tau - c.tpot) - hb) <= NB_REL * m.tau) d.nb |= NB_HEADROOM;
    }
  }
  // A candidate whose T membership rounding may change can change the
  // decision only if it is the choice, or if it is outside T and would come
  // first (or T is empty).  With a total order on T, flipping any set of
  // other unsure candidates leaves the choice where it is.  The random and
  // H-C-Q selectors depend on all of T.
  for (const Cand& c : A) {
    if (!c.unsure) continue;
    const bool decides = sel == SEL_RANDOM || sel == SEL_HCQ || &c == best ||
                         (!c.inT && (!best || before(sel, c, *best)));
    if (decides) d.nb |= (std::fabs(c.tpot - m.tau) <= NB_REL * m.tau) ? NB_TPOT : NB_TTFT;
  }
  d.flags = 0;
  if (!best) {
    if (m.flags & F_FALLBACK_DCQ) {
      // fallback by the D-C-Q key over the KVC-admissible set
      for (const Cand& c : A)
        if (c.inC && (!best || before(SEL_DCQ, c, *best))) best = &c;
    } else {
      // Cache-aware load balancing over the KVC-admissible set: the product
      // of pending uncached prefill tokens and active requests, both
      // counting the arriving request; ties to the lowest id.
      unsigned __int128 bestv = 0;
      for (const Cand& c : A) {
        if (!c.inC) continue;
        const unsigned __int128 v = lmetric(c);
        if (!best || v < bestv || (v == bestv && c.i < best->i)) {
          best = &c;
          bestv = v;
        }
      }
    }
    d.flags |= R_FALLBACK;
  }
  d.inst = best->i;
  d.hit = (int32_t)best->hit;
  d.ttft = best->ttft;
  d.tpot = best->tpot;
  if (best->ttft > slo) d.flags |= R_TTFT_MISS;
  if (!ttft_is_budget(*best) && std::fabs(best->ttft - slo) <= NB_REL * slo) d.nb |= NB_MISSFLAG;
  return d;
}

Chain chain_of(const uint64_t* pool, const int64_t* pre_off, const int32_t* pre_len,
               const int64_t* tail_off, const int32_t* tail_len, int32_t r) {
  return Chain{pool + pre_off[r], pre_len[r], pool + tail_off[r], tail_len[r]};
}

// Place one request on instance i (Sec. 7: the request path updates the
// instance's counters and its prefix tree as the request is routed): it
// joins the queue (Q += 1), its uncached tokens, measured against the set
// as it stands, join the pending prefill work, its tokens join the context
// sum, and its blocks enter the set in chain order until the cap is
// reached (refused blocks are counted in drop).  Returns the hit measured
// before the blocks enter.
int64_t commit_one(Snapshot& sn, const Chain& ch, int32_t i, int32_t block_tokens, int64_t& drop) {
  auto& set = sn.sets[(size_t)i];
  const int64_t L = (int64_t)ch.len() * block_tokens;
  const int64_t hitb = prefix_hit(set, ch);
  sn.Q[i] += 1;
  sn.P[i] += L - hitb * block_tokens;
  sn.S[i] += L;
  for (int32_t j = 0; j < ch.len(); ++j) {
    uint64_t key = ch.at(j);
    if (set.count(key)) continue;
    if ((int64_t)set.size() < sn.cap) set.insert(key);
    else ++drop;
  }
  return hitb;
}

}  // namespace

extern "C" {

// Build a snapshot: a hash set per instance from the CSR block lists, plus a
// copy of the load counters.  Returns 0, or -2 on allocation failure.
int orc_load(int32_t n_inst, int32_t cap, const int64_t* blk_off, const uint64_t* blk,
             const int32_t* D, const int32_t* Q, const int64_t* P, const int64_t* S, void** out) {
  *out = nullptr;
  Snapshot* sn = new (std::nothrow) Snapshot();
  if (!sn) return -2;
  try {
    sn->n_inst = n_inst;
    sn->cap = cap;
    sn->sets.resize((size_t)n_inst);
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t i = 0; i < n_inst; ++i) {
      auto& st = sn->sets[(size_t)i];
      st.reserve((size_t)(blk_off[i + 1] - blk_off[i]) * 2 + 16);
      for (int64_t k = blk_off[i]; k < blk_off[i + 1]; ++k) st.insert(blk[k]);
    }
    sn->D.assign(D, D + n_inst);
    sn->Q.assign(Q, Q + n_inst);
    sn->P.assign(P, P + n_inst);
    sn->S.assign(S, S + n_inst);
  } catch (const std::bad_alloc&) {
    delete sn;
    return -2;
  }
  *out = sn;
  return 0;
}

void orc_free(void* h) { delete static_cast<Snapshot*>(h); }

// Prefix hit of every request on every instance (no capacity test):
// hits[r * n_inst + i].
int orc_hits(void* h, const uint64_t* pool, const int64_t* pre_off, const int32_t* pre_len,
             const int64_t* tail_off, const int32_t* tail_len, int32_t n_req, uint32_t* hits,
             int32_t nthreads) {
  const Snapshot& sn = *static_cast<Snapshot*>(h);
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 16)
  for (int32_t r = 0; r < n_req; ++r) {
    Chain ch = chain_of(pool, pre_off, pre_len, tail_off, tail_len, r);
    for (int32_t i = 0; i < sn.n_inst; ++i)
      hits[(size_t)r * sn.n_inst + i] = (uint32_t)prefix_hit(sn.sets[(size_t)i], ch);
  }
  return 0;
}

// Algorithm 1 for every request of the window against the same snapshot.
// sizes (optional) receives |A|, |C|, |T| per request; nb (optional) the
// near-boundary bits.
int orc_score(void* h, const orc_model* m, const uint64_t* pool, const int64_t* pre_off,
              const int32_t* pre_len, const int64_t* tail_off, const int32_t* tail_len,
              int32_t n_req, int32_t* inst, int32_t* hit, double* ttft, double* tpot,
              uint32_t* flags, uint32_t* sizes, uint32_t* nb, int32_t nthreads) {
  const Snapshot& sn = *static_cast<Snapshot*>(h);
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 4)
  for (int32_t r = 0; r < n_req; ++r) {
    Chain ch = chain_of(pool, pre_off, pre_len, tail_off, tail_len, r);
    std::vector<Cand> A;
    Decision d = score_one(sn, *m, ch, A, r);
    inst[r] = d.inst;
    hit[r] = d.hit;
    ttft[r] = d.ttft;
    tpot[r] = d.tpot;
    flags[r] = d.flags;
    if (sizes) {
      sizes[3 * (size_t)r] = d.nA;
      sizes[3 * (size_t)r + 1] = d.nC;
      sizes[3 * (size_t)r + 2] = d.nT;
    }
    if (nb) nb[r] = d.nb;
  }
  return 0;
}

// Per-candidate detail of one request (for tests): for every instance,
// elig[i] = 1 if capacity-eligible; for those, hit, W, rho, TPOT, TTFT and
// C / T membership.  Returns the chosen instance (-1 on reject).
int orc_explain(void* h, const orc_model* m, const uint64_t* chain, int32_t len,
                uint8_t* elig, uint32_t* hit, double* W, double* rho, double* tpot,
                double* ttft, uint8_t* inC, uint8_t* inT) {
  const Snapshot& sn = *static_cast<Snapshot*>(h);
  Chain ch{chain, len, chain, 0};
  std::vector<Cand> A;
  Decision d = score_one(sn, *m, ch, A, 0);
  for (int32_t i = 0; i < sn.n_inst; ++i) {
    elig[i] = 0; hit[i] = 0; W[i] = rho[i] = tpot[i] = ttft[i] = 0.0; inC[i] = inT[i] = 0;
  }
  for (const Cand& c : A) {
    elig[c.i] = 1;
    hit[c.i] = (uint32_t)c.hit;
    W[c.i] = c.W;
    rho[c.i] = c.rho;
    tpot[c.i] = c.tpot;
    ttft[c.i] = c.ttft;
    inC[c.i] = c.inC;
    inT[c.i] = c.inT;
  }
  return d.inst;
}

// Apply decisions in array order: the arriving request joins the queue of
// its instance (Q += 1), adds its uncached tokens to the pending prefill
// work (measured against the table as left by the earlier entries), adds its
// tokens to the context sum, and its blocks enter the instance's set in
// chain order until the cap is reached.  Entries with instance -1 are
// skipped.  Returns the number of blocks refused at the cap in *dropped.
int orc_commit(void* h, const uint64_t* pool, const int64_t* pre_off, const int32_t* pre_len,
               const int64_t* tail_off, const int32_t* tail_len, const int32_t* inst, int32_t n,
               int32_t block_tokens, int64_t* dropped) {
  Snapshot& sn = *static_cast<Snapshot*>(h);
  int64_t drop = 0;
  for (int32_t k = 0; k < n; ++k) {
    const int32_t i = inst[k];
    if (i < 0) continue;
    Chain ch = chain_of(pool, pre_off, pre_len, tail_off, tail_len, k);
    (void)commit_one(sn, ch, i, block_tokens, drop);
  }
  *dropped = drop;
  return 0;
}

// Algorithm 1 per arrival: the requests are taken in array order; each is
// scored against the state left by the ones before it and, when placed,
// committed (as orc_commit) before the next one is scored.  Outputs as
// orc_score, plus the blocks refused at the cap in *dropped.  The snapshot
// is left in the final state.
//
// follow (optional): placements made by another implementation of the same
// schedule.  Where the oracle's own decision is near a boundary (rounding may
// decide it) and follow[r] differs, follow[r] is committed instead, so that
// both continue from the same state; it must be a capacity-eligible instance
// (else -1 is returned).  The outputs still hold the oracle's own decision.
int orc_schedule(void* h, const orc_model* m, const uint64_t* pool, const int64_t* pre_off,
                 const int32_t* pre_len, const int64_t* tail_off, const int32_t* tail_len,
                 int32_t n_req, int32_t* inst, int32_t* hit, double* ttft, double* tpot,
                 uint32_t* flags, uint32_t* sizes, uint32_t* nb, const int32_t* follow,
                 int64_t* dropped) {
  Snapshot& sn = *static_cast<Snapshot*>(h);
  int64_t drop = 0;
  std::vector<Cand> A;
  constexpr uint32_t NB_CHOICE = NB_RHO | NB_TPOT | NB_TTFT | NB_Z | NB_HEADROOM;
  for (int32_t r = 0; r < n_req; ++r) {
    Chain ch = chain_of(pool, pre_off, pre_len, tail_off, tail_len, r);
    const Decision d = score_one(sn, *m, ch, A, r);
    int32_t place = d.inst;
    if (follow && (d.nb & NB_CHOICE) && follow[r] != d.inst) {
      bool eligible = false;
      for (const Cand& c : A) eligible |= c.i == follow[r];
      if (!eligible) return -1;
      place = follow[r];
    }
    inst[r] = d.inst;
    hit[r] = d.hit;
    ttft[r] = d.ttft;
    tpot[r] = d.tpot;
    flags[r] = d.flags;
    if (sizes) {
      sizes[3 * (size_t)r] = d.nA;
      sizes[3 * (size_t)r + 1] = d.nC;
      sizes[3 * (size_t)r + 2] = d.nT;
    }
    if (nb) nb[r] = d.nb;
    if (place >= 0) (void)commit_one(sn, ch, place, m->block_tokens, drop);
  }
  *dropped = drop;
  return 0;
}

// Given placements applied in array order (entries with instance -1 are
// skipped): for each placed request, the hit, TTFT and TPOT its instance
// offers at its arrival, i.e. in the state left by the entries before it,
// then the commit of orc_commit.  Skipped entries get hit 0 and zero
// latencies.
int orc_replay(void* h, const orc_model* m, const uint64_t* pool, const int64_t* pre_off,
               const int32_t* pre_len, const int64_t* tail_off, const int32_t* tail_len,
               const int32_t* inst, int32_t n, int32_t* hit, double* ttft, double* tpot,
               int64_t* dropped) {
  Snapshot& sn = *static_cast<Snapshot*>(h);
  int64_t drop = 0;
  for (int32_t k = 0; k < n; ++k) {
    hit[k] = 0;
    ttft[k] = tpot[k] = 0.0;
    const int32_t i = inst[k];
    if (i < 0) continue;
    Chain ch = chain_of(pool, pre_off, pre_len, tail_off, tail_len, k);
    const int64_t L = (int64_t)ch.len() * m->block_tokens;
    const int64_t hb = prefix_hit(sn.sets[(size_t)i], ch);
    const int64_t c = hb * m->block_tokens;
    candidate_latency(sn, *m, i, L - c, c, L, tpot[k], ttft[k]);
    hit[k] = (int32_t)hb;
    (void)commit_one(sn, ch, i, m->block_tokens, drop);
  }
  *dropped = drop;
  return 0;
}

// Read back the load counters and set sizes.
int orc_state(void* h, int32_t* D, int32_t* Q, int64_t* P, int64_t* S, int64_t* set_size) {
  const Snapshot& sn = *static_cast<Snapshot*>(h);
  for (int32_t i = 0; i < sn.n_inst; ++i) {
    D[i] = sn.D[i];
    Q[i] = sn.Q[i];
    P[i] = sn.P[i];
    S[i] = sn.S[i];
    set_size[i] = (int64_t)sn.sets[(size_t)i].size();
  }
  return 0;
}

// Online calibration (Sec. 5.3): for each measured pure-decode forward, the
// factor of the segment of its batch size moves towards the
// measured-to-predicted ratio of the base model (no factor) with weight
// 0.02; the ratio is clipped to [0.5, 2] and the factor to [1, 2].  Samples
// with a non-positive base prediction carry no ratio and are skipped.
int orc_feedback_decode(orc_model* m, const int32_t* batch, const int64_t* ctx_tok,
                        const double* measured, int32_t n) {
  const double w = 0.02;
  for (int32_t k = 0; k < n; ++k) {
    const int s = segment_of(*m, batch[k]);
    const double pred = m->beta[s][0] + m->beta[s][1] * (double)batch[k] +
                        m->beta[s][2] * (double)ctx_tok[k];
    if (!(pred > 0.0)) continue;
    double ratio = measured[k] / pred;
    ratio = std::min(2.0, std::max(0.5, ratio));
    double f = (1.0 - w) * m->gamma[s] + w * ratio;
    m->gamma[s] = std::min(2.0, std::max(1.0, f));
  }
  return 0;
}

// Recent median output length: the lower median of the last (at most
// `window`) recorded lengths becomes the model's L_out.
int orc_feedback_output(void* h, orc_model* m, const int32_t* out_len, int32_t n, int32_t window) {
  Snapshot& sn = *static_cast<Snapshot*>(h);
  for (int32_t k = 0; k < n; ++k) sn.out_lens.push_back(out_len[k]);
  if (sn.out_lens.empty()) return 0;
  const size_t cnt = std::min(sn.out_lens.size(), (size_t)window);
  std::vector<int32_t> recent(sn.out_lens.end() - (long)cnt, sn.out_lens.end());
  std::sort(recent.begin(), recent.end());
  m->lout = (double)recent[(cnt - 1) / 2];
  return 0;
}

// Response-path transitions (Sec. 7: state follows the request and response
// paths).  kind 1: a queued request's first token (Q - 1, D + 1, P - tokens);
// 2: generated tokens of the decoding requests (S + tokens); 3: a decoding
// request finished (D - 1, S - tokens).  All or nothing: -5 if a counter
// would go negative, -1 on a bad kind or instance.
int orc_apply_events(void* h, const int32_t* inst, const int32_t* kind, const int64_t* tokens,
                     int32_t n) {
  Snapshot& sn = *static_cast<Snapshot*>(h);
  std::vector<int32_t> D = sn.D, Q = sn.Q;
  std::vector<int64_t> P = sn.P, S = sn.S;
  for (int32_t k = 0; k < n; ++k) {
    const int32_t i = inst[k];
    if (i < 0 || i >= sn.n_inst || tokens[k] < 0) return -1;
    if (kind[k] == 1) {
      Q[i] -= 1;
      D[i] += 1;
      P[i] -= tokens[k];
    } else if (kind[k] == 2) {
      S[i] += tokens[k];
    } else if (kind[k] == 3) {
      D[i] -= 1;
      S[i] -= tokens[k];
    } else {
      return -1;
    }
    if (D[i] < 0 || Q[i] < 0 || P[i] < 0 || S[i] < 0) return -5;
  }
  sn.D = D;
  sn.Q = Q;
  sn.P = P;
  sn.S = S;
  return 0;
}

int orc_max_threads(void) { return omp_get_max_threads(); }

}  // extern "C"
