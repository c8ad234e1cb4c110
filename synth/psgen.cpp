// Seeded synthetic scheduling-window generator.
//
// This module only draws inputs: chained block hashes for agent sessions,
// per-instance cached block sets, per-instance load counters and the
// latency-model coefficients.  It computes nothing the scheduler computes
// (no prefix match, no latency model, no filter, no selection).  Both the
// CPU oracle and the GPU library consume what it writes, and neither side
// shares any other code with the other.
//
// Workload shape (agentic traces, the paper's Sec. 3 and Table 2):
//   * a session has a base prefix of P_s blocks and grows by 8 blocks per
//     step for 8 steps (64 tail blocks);
//   * a request picks a session and a step k in 1..8 and asks for the first
//     P_s + 8k blocks of that session plus 1..F fresh blocks;
//   * a session's owner instance caches its first floor(u * (P_s + 64))
//     blocks, u ~ U[0.3, 1.0); sessions are inserted in a seeded random order
//     until the per-instance cap is reached, so every set stays closed under
//     prefixes;
//   * optionally a fraction of sessions starts with one shared system prompt.
//
// Hash chains: h_0 = 0 and h_j = splitmix64(h_{j-1} XOR id_j), where
// splitmix64(x) is the SplitMix64 output function applied to state x
// (Steele, Lea and Flood, OOPSLA 2014; Vigna's public-domain reference
// generator): z = x + 0x9E3779B97F4A7C15, then two xor-shift-multiply rounds
// and a final xor-shift.  The block ids id_j come from seeded SplitMix64
// streams.  A zero hash is never emitted (zero is the empty-slot sentinel of
// the GPU tables); the generator aborts with an error code if one ever
// appears.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

namespace {

inline uint64_t sm64_out(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// A SplitMix64 stream: state advances by the golden gamma, output = finaliser.
struct Stream {
  uint64_t s;
  Stream(uint64_t seed, uint64_t tag) : s(sm64_out(seed ^ sm64_out(tag))) {}
  uint64_t next() {
    uint64_t r = sm64_out(s);
    s += 0x9E3779B97F4A7C15ull;
    return r;
  }
  // Uniform integer in [a, b] (inclusive) by 128-bit multiply-high.
  int64_t uint_in(int64_t a, int64_t b) {
    if (b <= a) return a;
    unsigned __int128 range = (unsigned __int128)(uint64_t)(b - a) + 1u;
    unsigned __int128 p = (unsigned __int128)next() * range;
    return a + (int64_t)(uint64_t)(p >> 64);
  }
  // Uniform double in [0, 1).
  double u01() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
  double uniform(double a, double b) { return a + (b - a) * u01(); }
};

// Stream tags (arbitrary distinct constants, one per drawn quantity).
enum : uint64_t {
  T_SESS_LEN = 1, T_SESS_SP, T_SESS_IDS, T_SP_IDS, T_OWNER, T_OWNER_PERM,
  T_CACHE_U, T_INSERT_ORDER, T_REQ_SESS, T_REQ_PERM, T_REQ_STEP, T_REQ_FRESH,
  T_FRESH_IDS, T_LOAD, T_MODEL, T_SAT
};

// Zipf(s) over ranks 1..n by inverse CDF on the cumulative weights.
struct Zipf {
  std::vector<double> cdf;
  Zipf(int64_t n, double s) : cdf((size_t)n) {
    double acc = 0.0;
    for (int64_t k = 0; k < n; ++k) {
      acc += std::pow((double)(k + 1), -s);
      cdf[(size_t)k] = acc;
    }
  }
  int64_t draw(Stream& st) const {
    double u = st.u01() * cdf.back();
    auto it = std::upper_bound(cdf.begin(), cdf.end(), u);
    int64_t k = (int64_t)(it - cdf.begin());
    return k >= (int64_t)cdf.size() ? (int64_t)cdf.size() - 1 : k;
  }
};

void shuffle(std::vector<int32_t>& v, Stream& st) {
  for (int64_t i = (int64_t)v.size() - 1; i > 0; --i) {
    int64_t j = st.uint_in(0, i);
    std::swap(v[(size_t)i], v[(size_t)j]);
  }
}

}  // namespace

extern "C" {

// Generation parameters.  Every field is plain data; see the Python wrapper
// for the named workloads.
typedef struct {
  int32_t n_inst, n_req, n_sess;
  int32_t ps_min, ps_max;          // session base prefix P_s, blocks
  int32_t fresh_min, fresh_max;    // fresh blocks appended per request
  int32_t n_steps, step_blocks;    // 8 steps of 8 blocks
  int32_t owner_zipf;              // 0: uniform owner; 1: Zipf over permuted instances
  double owner_zipf_s;
  int32_t req_zipf;                // 0: uniform session; 1: Zipf over permuted sessions
  double req_zipf_s;
  double sp_frac;                  // fraction of sessions starting with the system prompt
  int32_t sp_blocks;               // system prompt length, blocks
  double cache_u_min, cache_u_max; // cached fraction of the full session chain
  int32_t cap;                     // per-instance cap on distinct cached blocks
  int32_t d_min, d_max;            // decoding requests per instance
  int32_t q_min, q_max;            // queued requests per instance
  int32_t ctx_min, ctx_max;        // context tokens per active request
  int64_t p_max;                   // pending prefill tokens when Q > 0
  double sat_frac;                 // fraction of "saturated" instances
  int32_t sat_d_min, sat_d_max;
  int64_t sat_s_min, sat_s_max;    // their total context tokens, drawn directly
  int32_t n_seg;                   // decode segments (<= 32)
  int32_t seg_ub[32];              // inclusive upper batch sizes
  int32_t gamma_unit_ub;           // segments with ub <= this get gamma = 1
  double gamma_min, gamma_max;     // gamma for the other segments
  double alpha_nom[6];             // nominal prefill coefficients
  double beta_nom[3];              // nominal decode coefficients
  double coef_jitter;              // coefficients = nominal * U[1-j, 1+j]
  uint64_t seed;
} psg_params;

struct psg_window {
  // pool: all session chains, then all fresh tails
  std::vector<uint64_t> pool;
  std::vector<int64_t> sess_off;
  std::vector<int32_t> sess_len, sess_base, sess_sp, sess_owner, sess_cached, sess_cached_eff;
  std::vector<int64_t> pre_off, tail_off;
  std::vector<int32_t> pre_len, tail_len, req_sess, req_step;
  std::vector<int64_t> blk_off;
  std::vector<uint64_t> blk;
  std::vector<int32_t> inst_sp_have;
  std::vector<int32_t> D, Q;
  std::vector<int64_t> P, S;
  float alpha[6];
  float beta[32][3];
  float gamma[32];
};

// Returns 0 on success, -1 on bad parameters, -2 on allocation failure,
// -3 if a zero hash was drawn.
int psg_generate(const psg_params* p, psg_window** out) {
  if (!p || !out) return -1;
  *out = nullptr;
  if (p->n_inst <= 0 || p->n_req < 0 || p->n_sess <= 0 || p->ps_min < 1 ||
      p->ps_max < p->ps_min || p->fresh_min < 0 || p->fresh_max < p->fresh_min ||
      p->n_steps < 1 || p->step_blocks < 0 || p->cap < 0 || p->n_seg < 1 ||
      p->n_seg > 32 || p->sp_blocks < 0)
    return -1;
  psg_window* w = new (std::nothrow) psg_window();
  if (!w) return -2;
  try {
    const uint64_t seed = p->seed;
    const int32_t tail_blocks = p->n_steps * p->step_blocks;
    const int32_t ns = p->n_sess;

    // ---- sessions: lengths, system-prompt membership, chains
    Stream s_len(seed, T_SESS_LEN), s_sp(seed, T_SESS_SP), s_ids(seed, T_SESS_IDS);
    Stream s_spids(seed, T_SP_IDS);
    std::vector<uint64_t> sp_ids((size_t)p->sp_blocks);
    for (auto& x : sp_ids) x = s_spids.next();
    w->sess_off.resize((size_t)ns);
    w->sess_len.resize((size_t)ns);
    w->sess_base.resize((size_t)ns);
    w->sess_sp.resize((size_t)ns);
    int64_t total = 0;
    for (int32_t s = 0; s < ns; ++s) {
      int32_t base = (int32_t)s_len.uint_in(p->ps_min, p->ps_max);
      w->sess_base[(size_t)s] = base;
      w->sess_len[(size_t)s] = base + tail_blocks;
      w->sess_sp[(size_t)s] = (p->sp_blocks > 0 && s_sp.u01() < p->sp_frac) ? 1 : 0;
      w->sess_off[(size_t)s] = total;
      total += base + tail_blocks;
    }
    // fresh tails are appended after the sessions
    Stream r_sess(seed, T_REQ_SESS), r_perm(seed, T_REQ_PERM), r_step(seed, T_REQ_STEP);
    Stream r_fresh(seed, T_REQ_FRESH), r_ids(seed, T_FRESH_IDS);
    const int32_t nr = p->n_req;
    w->pre_off.resize((size_t)nr);
    w->tail_off.resize((size_t)nr);
    w->pre_len.resize((size_t)nr);
    w->tail_len.resize((size_t)nr);
    w->req_sess.resize((size_t)nr);
    w->req_step.resize((size_t)nr);
    std::vector<int32_t> sess_perm((size_t)ns);
    for (int32_t s = 0; s < ns; ++s) sess_perm[(size_t)s] = s;
    shuffle(sess_perm, r_perm);
    Zipf* rz = p->req_zipf ? new Zipf(ns, p->req_zipf_s) : nullptr;
    int64_t fresh_total = 0;
    for (int32_t r = 0; r < nr; ++r) {
      int32_t s = rz ? sess_perm[(size_t)rz->draw(r_sess)] : (int32_t)r_sess.uint_in(0, ns - 1);
      int32_t k = (int32_t)r_step.uint_in(1, p->n_steps);
      int32_t f = (int32_t)r_fresh.uint_in(p->fresh_min, p->fresh_max);
      w->req_sess[(size_t)r] = s;
      w->req_step[(size_t)r] = k;
      w->pre_off[(size_t)r] = w->sess_off[(size_t)s];
      w->pre_len[(size_t)r] = w->sess_base[(size_t)s] + k * p->step_blocks;
      w->tail_len[(size_t)r] = f;
      fresh_total += f;
    }
    delete rz;
    w->pool.resize((size_t)(total + fresh_total));
    for (int32_t s = 0; s < ns; ++s) {
      uint64_t h = 0;
      uint64_t* dst = w->pool.data() + w->sess_off[(size_t)s];
      int32_t len = w->sess_len[(size_t)s];
      int32_t spn = w->sess_sp[(size_t)s] ? std::min(p->sp_blocks, w->sess_base[(size_t)s]) : 0;
      for (int32_t j = 0; j < len; ++j) {
        uint64_t id = j < spn ? sp_ids[(size_t)j] : s_ids.next();
        h = sm64_out(h ^ id);
        if (h == 0) { delete w; return -3; }
        dst[j] = h;
      }
    }
    int64_t cur = total;
    for (int32_t r = 0; r < nr; ++r) {
      int32_t f = w->tail_len[(size_t)r];
      w->tail_off[(size_t)r] = cur;
      int32_t s = w->req_sess[(size_t)r];
      uint64_t h = w->pool[(size_t)(w->pre_off[(size_t)r] + w->pre_len[(size_t)r] - 1)];
      for (int32_t j = 0; j < f; ++j) {
        h = sm64_out(h ^ r_ids.next());
        if (h == 0) { delete w; return -3; }
        w->pool[(size_t)(cur + j)] = h;
      }
      (void)s;
      cur += f;
    }

    // ---- owners and cached prefixes
    Stream o_st(seed, T_OWNER), o_perm(seed, T_OWNER_PERM), c_u(seed, T_CACHE_U);
    Stream ins(seed, T_INSERT_ORDER);
    std::vector<int32_t> inst_perm((size_t)p->n_inst);
    for (int32_t i = 0; i < p->n_inst; ++i) inst_perm[(size_t)i] = i;
    shuffle(inst_perm, o_perm);
    Zipf* oz = p->owner_zipf ? new Zipf(p->n_inst, p->owner_zipf_s) : nullptr;
    w->sess_owner.resize((size_t)ns);
    w->sess_cached.resize((size_t)ns);
    w->sess_cached_eff.resize((size_t)ns);
    for (int32_t s = 0; s < ns; ++s) {
      w->sess_owner[(size_t)s] =
          oz ? inst_perm[(size_t)oz->draw(o_st)] : (int32_t)o_st.uint_in(0, p->n_inst - 1);
      double u = c_u.uniform(p->cache_u_min, p->cache_u_max);
      int32_t cl = (int32_t)std::floor(u * (double)w->sess_len[(size_t)s]);
      w->sess_cached[(size_t)s] = std::min(cl, w->sess_len[(size_t)s]);
    }
    delete oz;
    std::vector<int32_t> order((size_t)ns);
    for (int32_t s = 0; s < ns; ++s) order[(size_t)s] = s;
    shuffle(order, ins);
    std::vector<int32_t> count((size_t)p->n_inst, 0);
    w->inst_sp_have.assign((size_t)p->n_inst, 0);
    // per-instance list of (session, start, end) ranges inserted, in insertion order
    std::vector<std::vector<int64_t>> ranges((size_t)p->n_inst);
    for (int32_t s : order) {
      int32_t i = w->sess_owner[(size_t)s];
      int32_t cl = w->sess_cached[(size_t)s];
      int32_t spn = w->sess_sp[(size_t)s] ? std::min(p->sp_blocks, w->sess_base[(size_t)s]) : 0;
      // blocks [0, start) are already present (shared system prompt)
      int32_t start = spn > 0 ? std::min(w->inst_sp_have[(size_t)i], cl) : 0;
      int32_t room = p->cap - count[(size_t)i];
      int32_t take = std::max(0, std::min(cl - start, room));
      w->sess_cached_eff[(size_t)s] = start + take;
      if (take > 0) {
        ranges[(size_t)i].push_back(w->sess_off[(size_t)s] + start);
        ranges[(size_t)i].push_back(take);
        count[(size_t)i] += take;
      }
      if (spn > 0)
        w->inst_sp_have[(size_t)i] =
            std::max(w->inst_sp_have[(size_t)i], std::min(start + take, spn));
    }
    w->blk_off.resize((size_t)p->n_inst + 1);
    int64_t nb = 0;
    for (int32_t i = 0; i < p->n_inst; ++i) {
      w->blk_off[(size_t)i] = nb;
      nb += count[(size_t)i];
    }
    w->blk_off[(size_t)p->n_inst] = nb;
    w->blk.resize((size_t)nb);
    for (int32_t i = 0; i < p->n_inst; ++i) {
      uint64_t* dst = w->blk.data() + w->blk_off[(size_t)i];
      const auto& rg = ranges[(size_t)i];
      for (size_t k = 0; k < rg.size(); k += 2) {
        std::memcpy(dst, w->pool.data() + rg[k], (size_t)rg[k + 1] * sizeof(uint64_t));
        dst += rg[k + 1];
      }
    }

    // ---- load state
    Stream ld(seed, T_LOAD), sat(seed, T_SAT);
    w->D.resize((size_t)p->n_inst);
    w->Q.resize((size_t)p->n_inst);
    w->P.resize((size_t)p->n_inst);
    w->S.resize((size_t)p->n_inst);
    for (int32_t i = 0; i < p->n_inst; ++i) {
      bool is_sat = p->sat_frac > 0.0 && sat.u01() < p->sat_frac;
      int32_t d = is_sat ? (int32_t)ld.uint_in(p->sat_d_min, p->sat_d_max)
                         : (int32_t)ld.uint_in(p->d_min, p->d_max);
      int32_t q = (int32_t)ld.uint_in(p->q_min, p->q_max);
      int64_t s = 0;
      if (is_sat) {
        s = ld.uint_in(p->sat_s_min, p->sat_s_max);
      } else {
        for (int32_t a = 0; a < d + q; ++a) s += ld.uint_in(p->ctx_min, p->ctx_max);
      }
      int64_t pend = q > 0 ? ld.uint_in(0, p->p_max) : 0;
      w->D[(size_t)i] = d;
      w->Q[(size_t)i] = q;
      w->S[(size_t)i] = s;
      w->P[(size_t)i] = pend;
    }

    // ---- model coefficients (stored in fp32, the interface precision)
    Stream md(seed, T_MODEL);
    const double j = p->coef_jitter;
    for (int k = 0; k < 6; ++k) w->alpha[k] = (float)(p->alpha_nom[k] * md.uniform(1.0 - j, 1.0 + j));
    for (int s = 0; s < 32; ++s) {
      for (int k = 0; k < 3; ++k) w->beta[s][k] = 0.0f;
      w->gamma[s] = 1.0f;
    }
    for (int s = 0; s < p->n_seg; ++s) {
      for (int k = 0; k < 3; ++k) w->beta[s][k] = (float)(p->beta_nom[k] * md.uniform(1.0 - j, 1.0 + j));
      w->gamma[s] = p->seg_ub[s] <= p->gamma_unit_ub ? 1.0f
                                                     : (float)md.uniform(p->gamma_min, p->gamma_max);
    }
  } catch (const std::bad_alloc&) {
    delete w;
    return -2;
  }
  *out = w;
  return 0;
}

void psg_free(psg_window* w) { delete w; }

// Sizes: pool, blocks, sessions, requests, instances.
void psg_sizes(const psg_window* w, int64_t* sz) {
  sz[0] = (int64_t)w->pool.size();
  sz[1] = (int64_t)w->blk.size();
  sz[2] = (int64_t)w->sess_off.size();
  sz[3] = (int64_t)w->pre_off.size();
  sz[4] = (int64_t)w->D.size();
}

// Field accessors: pointers stay valid until psg_free.
const void* psg_field(const psg_window* w, const char* name) {
#define F(n) if (!std::strcmp(name, #n)) return w->n.data();
  F(pool) F(sess_off) F(sess_len) F(sess_base) F(sess_sp) F(sess_owner) F(sess_cached)
  F(sess_cached_eff) F(pre_off) F(tail_off) F(pre_len) F(tail_len) F(req_sess) F(req_step)
  F(blk_off) F(blk) F(inst_sp_have) F(D) F(Q) F(P) F(S)
#undef F
  if (!std::strcmp(name, "alpha")) return w->alpha;
  if (!std::strcmp(name, "beta")) return w->beta;
  if (!std::strcmp(name, "gamma")) return w->gamma;
  return nullptr;
}

// The SplitMix64 output function, exported so that tests can rebuild chains.
uint64_t psg_splitmix64(uint64_t x) { return sm64_out(x); }

}  // extern "C"
