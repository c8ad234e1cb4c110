// Per-arrival scheduler (Algorithm 1 taken one request at a time, each
// placement committed before the next request is scored): one workgroup
// walks a launch's requests in order.  See seq_kernel below.

#include "ps_common.h"

namespace {

// ----------------------------------------------------- per-arrival scheduler
// One wave's share of a workgroup-wide reduction.
struct SeqPart {
  uint64_t keyT, keyF;
  uint32_t hroom, nC, nT, wmin, nA, pad;
};

// One wave's share of the check of a speculative result (below).
struct FastPart {
  uint64_t keyT, keyF;  // least selector / fallback key over the changed instances in T / C
  uint32_t conf;        // a changed instance now holds the block where the hit stopped
  uint32_t wb, wc;      // least W over the changed instances eligible then / now
  uint32_t eb, ec;      // changed instances eligible then / now
  uint32_t cb, cc;      // ... in C then / now
  uint32_t tb, tc;      // ... in T then / now
  uint32_t pad;
};

// Workgroup LDS of the scheduler (a fixed layout, plus the dirty bitmap).
struct SeqShared {
  uint64_t stage[kSeqStage];          // the request's chain head
  SeqPart part[2][kSeqWaves];         // reduction partials (alternating)
  FastPart fp[kSeqWaves];
  uint32_t cnt[kSeqU][kSeqWaves];     // per-wave counts of one insert step
  uint32_t ext[kExtMax][2];           // hit extensions: instance, first unknown position
  uint32_t ring[3];                   // first-absent minima of the sweeps
  uint32_t n_ext, hit, pick, count;
  int64_t rp;                         // row position found by a run walk's probe
  // instances placed on in this launch (the dirty ones), in order, with
  // their state at the launch's start
  uint32_t n_u;
  uint32_t n_fast, n_full;            // decisions from speculation / scored in full
  uint32_t u_id[kSpecBatch];
  InstState u_old[kSpecBatch];
};

__device__ __forceinline__ uint64_t seq_key(const SeqShared& sh, const ChainRef& c, int32_t j) {
  return j < kSeqStage ? sh.stage[j] : chain_global(c, j);
}

// The request's chain head into LDS, eight loads in flight per thread.
// Visible after the next barrier.
__device__ __forceinline__ void stage_chain(SeqShared& sh, const ChainRef& c, int tid, int NT) {
  const int32_t nst = c.len < kSeqStage ? c.len : kSeqStage;
  for (int32_t j0 = 0; j0 < nst; j0 += 8 * NT) {
    uint64_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int32_t j = j0 + u * NT + tid;
      v[u] = j < nst ? chain_global(c, j) : 0ull;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int32_t j = j0 + u * NT + tid;
      if (j < nst) sh.stage[j] = v[u];
    }
  }
}

// Key of the first of the n listed entries whose instance is not marked in
// `dirty`, or ~0 when there is none (every lane of the wave gets it).  Lane
// l holds the key of entry l (the lists have at most 64 entries).
__device__ __forceinline__ uint64_t spec_first_outside(uint64_t k, uint32_t n,
                                                       const uint64_t* dirty, int lane) {
  static_assert(kSpecList == 64, "one list entry per lane");
  const bool out = (uint32_t)lane < n && !test_bit(dirty, (uint32_t)(k & 0xFFFFu));
  const uint64_t bm = __ballot(out);
  if (bm == 0ull) return ~0ull;
  return (uint64_t)lane_value64((int64_t)k, __builtin_ctzll(bm));
}

// First position at or after `pos` whose block instance i does not hold,
// given that it holds every block before `pos`: each step probes blockDim.x
// x kSeqU positions at once (one bucket load per position in flight) and
// takes the first absent one by a workgroup minimum through a ring of three
// LDS slots (one barrier per step).  Workgroup-uniform arguments; a barrier
// must separate two calls.
__device__ uint32_t seq_sweep(const Tables& t, uint32_t i, const ChainRef& c, SeqShared& sh,
                              int32_t pos) {
  const int tid = threadIdx.x, NT = blockDim.x;
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, i);
  if (tid == 0) sh.ring[0] = sh.ring[1] = sh.ring[2] = ~0u;
  __syncthreads();
  for (int it = 0; pos < ell; ++it, pos += NT * kSeqU) {
    uint64_t key[kSeqU];
    Bucket bk[kSeqU];
#pragma unroll
    for (int u = 0; u < kSeqU; ++u) {
      const int32_t j = pos + u * NT + tid;
      key[u] = j < ell ? seq_key(sh, c, j) : 0ull;
      if (key[u] != 0ull)
        bk[u] = load_bucket(tab + (size_t)bucket_of(key[u], i, t.shift) * kSlotsPerBucket);
    }
    uint32_t first = ~0u;
#pragma unroll
    for (int u = 0; u < kSeqU; ++u) {
      const int32_t j = pos + u * NT + tid;
      if (j >= ell) continue;
      bool f = false, e = false;
      if (key[u] != 0ull) {
#pragma unroll
        for (int s = 0; s < kSlotsPerBucket; ++s) {
          f |= bk[u].k[s] == key[u];
          e |= bk[u].k[s] == 0ull;
        }
        if (!f && !e) f = probe(t, i, key[u]);  // bucket full: follow the probe sequence
      }
      if (!f && (uint32_t)j < first) first = (uint32_t)j;
    }
    uint32_t* slot = &sh.ring[it % 3];
    if (first != ~0u) atomicMin(slot, first);
    __syncthreads();
    const uint32_t m = *slot;
    if (tid == 0) sh.ring[(it + 2) % 3] = ~0u;  // read last in the previous step, written next in two
    if (m != ~0u) return m;
  }
  return (uint32_t)ell;
}

// Row position of `key` in instance i's row, or -1 when the instance does
// not hold it (one thread).
__device__ int64_t probe_rowpos(const Tables& t, uint32_t i, uint64_t key) {
  if (key == 0) return -1;
  const uint64_t* tab = table_of(t, i);
  uint32_t b = bucket_of(key, i, t.shift);
  for (uint32_t step = 0; step <= t.bmask; ++step) {
    const Bucket bk = load_bucket(tab + (size_t)b * kSlotsPerBucket);
    bool e = false;
#pragma unroll
    for (int s = 0; s < kSlotsPerBucket; ++s) {
      if (bk.k[s] == key) return t.rowpos[(size_t)i * t.slots + (size_t)b * kSlotsPerBucket + s];
      e |= bk.k[s] == 0;
    }
    if (e) return -1;
    b = (b + 1) & t.bmask;
  }
  return -1;
}

// Hit extension along instance i's row: the block at `pos` is probed (one
// thread) and the chain after it is compared with the row after it, 16
// positions per thread per step (coalesced row reads, the chain from LDS),
// the first mismatch by a workgroup minimum; a mismatch is probed again, as
// it may start another run of the row.  A run shorter than 8 blocks hands
// the rest to seq_sweep.  Requires every block before `pos` to be held;
// workgroup-uniform arguments; a barrier must separate two calls.
__device__ uint32_t seq_run_walk(const Tables& t, uint32_t i, const ChainRef& c, SeqShared& sh,
                                 int32_t pos) {
  constexpr int kRunU = 16;
  const int tid = threadIdx.x, NT = blockDim.x;
  const int32_t ell = c.len;
  const uint64_t* row = t.rows + (size_t)i * (size_t)t.row_cap;
  const int64_t rlen = t.count[i];
  while (pos < ell) {
    if (tid == 0) {
      sh.rp = probe_rowpos(t, i, seq_key(sh, c, pos));
      sh.ring[0] = sh.ring[1] = sh.ring[2] = ~0u;
    }
    __syncthreads();
    const int64_t rp = sh.rp;
    if (rp < 0) return (uint32_t)pos;
    const int32_t start = pos + 1;
    int32_t next = -1;
    for (int it = 0; next < 0; ++it) {
      const int32_t q = start + it * NT * kRunU;
      if (q >= ell) return (uint32_t)ell;
      const int64_t k = rp + 1 + (int64_t)it * NT * kRunU;
      uint64_t rk[kRunU];
#pragma unroll
      for (int u = 0; u < kRunU; ++u) {
        const int32_t j = q + u * NT + tid;
        const int64_t kk = k + u * NT + tid;
        rk[u] = (j < ell && kk < rlen) ? row[kk] : 0ull;
      }
      uint32_t first = ~0u;
#pragma unroll
      for (int u = 0; u < kRunU; ++u) {
        const int32_t j = q + u * NT + tid;
        const int64_t kk = k + u * NT + tid;
        if (j < ell && (kk >= rlen || seq_key(sh, c, j) != rk[u]) && (uint32_t)j < first)
          first = (uint32_t)j;
      }
      uint32_t* slot = &sh.ring[it % 3];
      if (first != ~0u) atomicMin(slot, first);
      __syncthreads();
      const uint32_t m = *slot;
      if (tid == 0) sh.ring[(it + 2) % 3] = ~0u;
      if (m != ~0u) next = (int32_t)m;
    }
    __syncthreads();  // ring and rp are rewritten by the next probe
    if (next - start < 8) return seq_sweep(t, i, c, sh, next);
    pos = next;
  }
  return (uint32_t)ell;
}

// Algorithm 1 per arrival (each placement changes the state the next
// request is scored against).  One workgroup takes the launch's requests in
// order; thread t owns the instances t, t + blockDim.x, ...  Per request:
//  (1) the capacity guard and |A| (a request with A empty is rejected
//      without touching any table; one longer than every room seen by the
//      last capacity pass, without a pass);
//  (2) live hits of the eligible instances: the hit at the launch's start,
//      extended where an instance that took a request earlier in the launch
//      now holds the next block (one probe per such instance, then a walk
//      of the whole workgroup along the instance's row);
//  (3) W_min, then C, T and the selector's key exactly as the window kernel
//      evaluates them, each reduced over the workgroup (every thread
//      combines the waves' partials, so all of them hold the decision);
//  (4) the owner of the chosen instance writes the result and moves the
//      instance's counters; the workgroup inserts the request's new blocks
//      into the instance's table and row in chain order (when the cap might
//      bind, wave 0 does it position by position to refuse exactly the
//      blocks past the cap).
// The next request starts after a workgroup barrier, so its probes see
// those inserts.  Replay (a.forced): the given instance is
// measured and committed, without (1) and (3).
__global__ __launch_bounds__(kSeqMaxThreads) void seq_kernel(SeqArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  SeqShared& sh = *reinterpret_cast<SeqShared*>(smem);
  uint64_t* dirty = reinterpret_cast<uint64_t*>(smem + sizeof(SeqShared));
  const int32_t n_inst = a.n_inst;
  const int32_t nw = (n_inst + 63) >> 6;
  const int tid = threadIdx.x;
  const int NT = blockDim.x;
  const int lane = tid & 63, wv = tid >> 6, nwv = NT >> 6;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  const DevModel& m = *a.model;
  const bool replay = a.forced != nullptr;
  ScoreArgs sa{};
  sa.inst = a.inst;
  for (int32_t w = tid; w < nw; w += NT) dirty[w] = 0ull;
  if (tid == 0) sh.n_u = sh.n_fast = sh.n_full = 0u;
  unsigned long long drop = 0;
  int pb = 0;  // partial buffer of the next reduction (alternates)
  ps_req qn = a.reqs[a.r0];
  // Largest capacity room (M_KV - S over instances with A + 1 <= B_max)
  // seen by the last capacity pass.  Rooms only shrink during a launch, so
  // a request longer than it has A empty without another pass.
  int64_t room_ub = INT64_MAX;

  for (int32_t r = a.r0; r < a.r1; ++r) {
    // The previous request's inserts, rows and counters.  Only this
    // workgroup touches the tables during the launch, so workgroup scope is
    // enough: the waves share one CU and its L1.
    __syncthreads();
    const ps_req q = qn;
    if (r + 1 < a.r1) qn = a.reqs[r + 1];  // in flight while this request runs
    if (!req_valid(q, a.pool_len)) {
      if (tid == 0) {
        a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_INVALID};
        if (a.sizes) a.sizes[3 * (size_t)r] = a.sizes[3 * (size_t)r + 1] = a.sizes[3 * (size_t)r + 2] = 0;
      }
      continue;
    }
    const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
    const int32_t ell = c.len;
    const int64_t L = (int64_t)ell * m.bs;
    const float Lf = (float)L;
    uint32_t* H = a.hits + (size_t)(r - a.r0) * (size_t)n_inst;
    const int32_t forced = replay ? a.forced[r] : -1;

    int32_t best = -1;
    uint32_t fl = PS_R_REJECT, nA = 0, nC = 0, nT = 0;
    const float Z = recompute_raw(m, Lf, Lf);  // T_pf(L, 0) - T_pf(0, L)
    const float tpf_cold = t_prefill(m, Lf, 0.0f);
    const float slo = fmaxf(m.ttft_floor, tpf_cold);
    const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
    bool staged = false, fast = false;

    // (0) the speculative result: scored against the launch's starting
    // state, it still decides the request unless an instance placed on
    // since then (the set U) changes W_min or the choice
    if (a.spec != nullptr && !replay) {
      const SpecRec& sp = a.spec[r - a.r0];
      stage_chain(sh, c, tid, NT);  // the commit reads it
      const uint64_t lt_key = sp.lt[lane].key;  // read before n is known
      staged = true;
      const uint32_t n_u = sh.n_u;
      const uint32_t wmin_b = sp.wmin;
      const float wmin = __uint_as_float(wmin_b);
      FastPart f{~0ull, ~0ull, 0u, ~0u, ~0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
      for (uint32_t k = (uint32_t)tid; k < n_u; k += (uint32_t)NT) {
        const uint32_t u = sh.u_id[k];
        const InstState so = sh.u_old[k];  // as the speculative scoring saw it
        const InstState sc = a.inst[u];    // now
        const uint32_t h = H[u];           // its hit then
        const bool eb = eligible(m, so.A1, so.S, L), ec = eligible(m, sc.A1, sc.S, L);
        // the hit still stops at h unless u has taken the block at h since
        if (ec && (int32_t)h < ell && probe(a.t, u, chain_global(c, (int32_t)h))) f.conf = 1u;
        const uint32_t wb = __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)h * m.bs), Lf)));
        const bool cpass = !kvc || (__uint_as_float(wb) - wmin) / Z <= m.eta;
        if (eb) {
          f.eb += 1u;
          f.wb = wb < f.wb ? wb : f.wb;
          if (cpass) {
            f.cb += 1u;
            if (a.sizes)
              f.tb += member_with(m, [&]() { return so; }, h, L, Lf, wmin, Z, kvc, slo).inT ? 1u : 0u;
          }
        }
        if (ec) {
          f.ec += 1u;
          f.wc = wb < f.wc ? wb : f.wc;
          const Member mb = member_with(m, [&]() { return sc; }, h, L, Lf, wmin, Z, kvc, slo);
          if (mb.inC) {
            f.cc += 1u;
            const uint64_t lm = (uint64_t)(mb.st.P + mb.n_tok) * (uint64_t)mb.st.A1;
            const uint64_t kf = (m.flags & PS_F_FALLBACK_DCQ) ? dcq_key(mb.st, h, u) : ((lm << 16) | u);
            f.keyF = kf < f.keyF ? kf : f.keyF;
            if (mb.inT) {
              f.tc += 1u;
              const uint64_t kt = select_key(m.sel, mb.st, h, u, lm);
              f.keyT = kt < f.keyT ? kt : f.keyT;
            }
          }
        }
      }
      {
        FastPart w;
        w.keyT = wave_min_u64(f.keyT);
        w.keyF = wave_min_u64(f.keyF);
        w.conf = __ballot(f.conf != 0u) ? 1u : 0u;
        w.wb = wave_min_u32(f.wb);
        w.wc = wave_min_u32(f.wc);
        w.eb = wave_sum_u32(f.eb);
        w.ec = wave_sum_u32(f.ec);
        w.cb = wave_sum_u32(f.cb);
        w.cc = wave_sum_u32(f.cc);
        w.tb = wave_sum_u32(f.tb);
        w.tc = wave_sum_u32(f.tc);
        w.pad = 0u;
        if (lane == 0) sh.fp[wv] = w;
      }
      __syncthreads();
      FastPart g = sh.fp[0];
      for (int k = 1; k < nwv; ++k) {
        const FastPart& p = sh.fp[k];
        g.keyT = p.keyT < g.keyT ? p.keyT : g.keyT;
        g.keyF = p.keyF < g.keyF ? p.keyF : g.keyF;
        g.conf |= p.conf;
        g.wb = p.wb < g.wb ? p.wb : g.wb;
        g.wc = p.wc < g.wc ? p.wc : g.wc;
        g.eb += p.eb;
        g.ec += p.ec;
        g.cb += p.cb;
        g.cc += p.cc;
        g.tb += p.tb;
        g.tc += p.tc;
      }
      const uint32_t nA_now = sp.nA - g.eb + g.ec;
      // W_min is unchanged unless a hit moved (conf) or the only changed
      // instances at the minimum all left A: then it is not known here
      bool ok = g.conf == 0u && !(g.wb == wmin_b && g.wc != wmin_b) && g.wc >= wmin_b;
      if (ok && nA_now > 0u) {
        // the other members of T and C are as speculated; the first listed
        // one outside U is the least of them when the list shows it
        const uint64_t t0 = spec_first_outside(lt_key, sp.nLT, dirty, lane);
        if (t0 == ~0ull && sp.nLT < sp.nT) {
          ok = false;
        } else {
          const uint64_t kT = t0 < g.keyT ? t0 : g.keyT;
          if (kT != ~0ull) {
            best = (int32_t)(kT & 0xFFFFu);
            fl = 0;
          } else {
            const uint64_t f0 = spec_first_outside(sp.lf[lane].key, sp.nLF, dirty, lane);
            if (f0 == ~0ull && sp.nLF < sp.nC) {
              ok = false;
            } else {
              const uint64_t kF = f0 < g.keyF ? f0 : g.keyF;
              if (kF != ~0ull) {
                best = (int32_t)(kF & 0xFFFFu);
                fl = PS_R_FALLBACK;
              }
            }
          }
        }
      }
      if (ok) {
        fast = true;
        nA = nA_now;
        if (nA_now > 0u) {
          nC = sp.nC - g.cb + g.cc;
          nT = sp.nT - g.tb + g.tc;
        }
      } else {
        best = -1;
        fl = PS_R_REJECT;
      }
      if (tid == 0) {
        if (fast) sh.n_fast += 1u;
        else sh.n_full += 1u;
      }
    }

    if (!fast) {
    // (1) capacity guard
    if (!replay && L <= room_ub) {
      uint32_t al = 0;
      uint64_t rl = ~0ull;  // ~(room + 1), minimised (room >= -1)
      for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
        InstState st[kSeqB];
#pragma unroll
        for (int u = 0; u < kSeqB; ++u) {
          const int32_t i = base + u * NT + tid;
          if (i < n_inst) st[u] = a.inst[i];
        }
#pragma unroll
        for (int u = 0; u < kSeqB; ++u) {
          if (base + u * NT + tid >= n_inst) continue;
          al += eligible(m, st[u].A1, st[u].S, L) ? 1u : 0u;
          const int64_t room = st[u].A1 <= m.b_max ? m.kv_cap - st[u].S : -1;
          const uint64_t x = ~((uint64_t)room + 1ull);
          rl = x < rl ? x : rl;
        }
      }
      al = wave_sum_u32(al);
      rl = wave_min_u64(rl);
      if (lane == 0) {
        sh.part[pb][wv].nA = al;
        sh.part[pb][wv].keyF = rl;
      }
      __syncthreads();
      uint64_t rmin = ~0ull;
      for (int k = 0; k < nwv; ++k) {
        nA += sh.part[pb][k].nA;
        rmin = sh.part[pb][k].keyF < rmin ? sh.part[pb][k].keyF : rmin;
      }
      pb ^= 1;
      room_ub = (int64_t)(~rmin - 1ull);
    }
    const bool work = replay ? forced >= 0 : nA > 0;
    if (work) {
      // (2) live hits
      if (!staged) stage_chain(sh, c, tid, NT);
      if (tid == 0) sh.n_ext = 0u;
      __syncthreads();
      for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
        // instances that took a request in this launch, are eligible and
        // whose hit stopped before the end of the chain: probe the block
        // the hit stopped at (the loads of a batch in flight together)
        bool cand[kSeqB];
        uint32_t vv[kSeqB];
#pragma unroll
        for (int u = 0; u < kSeqB; ++u) {
          const int32_t i = base + u * NT + tid;
          cand[u] = i < n_inst && test_bit(dirty, (uint32_t)i) && (!replay || i == forced);
          vv[u] = 0;
          if (cand[u]) {
            const InstState st = a.inst[i];
            vv[u] = H[i];
            cand[u] = (replay || eligible(m, st.A1, st.S, L)) && (int32_t)vv[u] < ell;
          }
        }
        uint64_t key[kSeqB];
        Bucket bk[kSeqB];
#pragma unroll
        for (int u = 0; u < kSeqB; ++u) {
          const int32_t i = base + u * NT + tid;
          key[u] = cand[u] ? seq_key(sh, c, (int32_t)vv[u]) : 0ull;
          if (key[u] != 0ull)
            bk[u] = load_bucket(table_of(a.t, (uint32_t)i) +
                                (size_t)bucket_of(key[u], (uint32_t)i, a.t.shift) * kSlotsPerBucket);
        }
#pragma unroll
        for (int u = 0; u < kSeqB; ++u) {
          const int32_t i = base + u * NT + tid;
          if (key[u] == 0ull) continue;
          bool f = false, emp = false;
#pragma unroll
          for (int sl = 0; sl < kSlotsPerBucket; ++sl) {
            f |= bk[u].k[sl] == key[u];
            emp |= bk[u].k[sl] == 0ull;
          }
          if (!f && !emp) f = probe(a.t, (uint32_t)i, key[u]);
          if (!f) continue;
          const uint32_t v = vv[u];
        const uint32_t e = atomicAdd(&sh.n_ext, 1u);
        if (e < kExtMax) {
          sh.ext[e][0] = (uint32_t)i;
          sh.ext[e][1] = v + 1u;
        } else {  // beyond the list: walk it alone
          uint32_t h = v + 1u;
          while ((int32_t)h < ell && probe(a.t, (uint32_t)i, seq_key(sh, c, (int32_t)h))) ++h;
          H[i] = h;
        }
        }
      }
      __syncthreads();
      const uint32_t n_ext = sh.n_ext < kExtMax ? sh.n_ext : kExtMax;
      for (uint32_t e = 0; e < n_ext; ++e) {
        const uint32_t i = sh.ext[e][0];
        const uint32_t h = seq_run_walk(a.t, i, c, sh, (int32_t)sh.ext[e][1]);
        if (tid == 0) H[i] = h;
        __syncthreads();
      }

      if (replay) {
        best = forced;
        fl = 0;
      } else {
        // (3a) minimum recomputation penalty over A
        uint32_t wl = 0x7F800000u;
        for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
          InstState st[kSeqB];
          uint32_t hv[kSeqB];
#pragma unroll
          for (int u = 0; u < kSeqB; ++u) {
            const int32_t i = base + u * NT + tid;
            if (i < n_inst) {
              st[u] = a.inst[i];
              hv[u] = H[i];
            }
          }
#pragma unroll
          for (int u = 0; u < kSeqB; ++u) {
            if (base + u * NT + tid >= n_inst || !eligible(m, st[u].A1, st[u].S, L)) continue;
            const float W = fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)hv[u] * m.bs), Lf));
            const uint32_t wb = __float_as_uint(W);
            wl = wb < wl ? wb : wl;
          }
        }
        wl = (uint32_t)wave_min_u64((uint64_t)wl);
        if (lane == 0) sh.part[pb][wv].wmin = wl;
        __syncthreads();
        uint32_t wmin_bits = 0x7F800000u;
        for (int k = 0; k < nwv; ++k) {
          const uint32_t x = sh.part[pb][k].wmin;
          wmin_bits = x < wmin_bits ? x : wmin_bits;
        }
        pb ^= 1;
        const float wmin = __uint_as_float(wmin_bits);

        // (3b) filters and keys
        Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
        for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
          InstState st[kSeqB];
          uint32_t hv[kSeqB];
#pragma unroll
          for (int u = 0; u < kSeqB; ++u) {
            const int32_t i = base + u * NT + tid;
            if (i < n_inst) {
              st[u] = a.inst[i];
              hv[u] = H[i];
            }
          }
#pragma unroll
          for (int u = 0; u < kSeqB; ++u) {
            const int32_t i = base + u * NT + tid;
            if (i >= n_inst || !eligible(m, st[u].A1, st[u].S, L)) continue;
            const InstState su = st[u];
            evaluate_with(m, acc, (uint32_t)i, hv[u], [&]() { return su; }, L, Lf, wmin, Z, kvc,
                          slo);
          }
        }
        uint64_t kT;
        uint32_t hr = ~0u;
        if (m.sel == PS_SEL_HCQ) {
          const uint64_t hmin = wave_min_u64((uint64_t)acc.hroom);
          kT = wave_min_u64((uint64_t)acc.hroom == hmin ? acc.keyT : ~0ull);
          hr = (uint32_t)hmin;
        } else {
          kT = wave_min_u64(acc.keyT);
        }
        const uint64_t kF = wave_min_u64(acc.keyF);
        const uint32_t cC = wave_sum_u32(acc.nC);
        const uint32_t cT = wave_sum_u32(acc.nT);
        if (lane == 0) {
          SeqPart& p = sh.part[pb][wv];
          p.keyT = kT;
          p.keyF = kF;
          p.hroom = hr;
          p.nC = cC;
          p.nT = cT;
        }
        __syncthreads();
        uint64_t keyT = ~0ull, keyF = ~0ull;
        uint32_t hroom = ~0u;
        for (int k = 0; k < nwv; ++k) {
          const SeqPart& p = sh.part[pb][k];
          if (m.sel == PS_SEL_HCQ) {
            if (p.hroom < hroom || (p.hroom == hroom && p.keyT < keyT)) {
              hroom = p.hroom;
              keyT = p.keyT;
            }
          } else {
            keyT = p.keyT < keyT ? p.keyT : keyT;
          }
          keyF = p.keyF < keyF ? p.keyF : keyF;
          nC += p.nC;
          nT += p.nT;
        }
        pb ^= 1;

        if (m.sel == PS_SEL_RANDOM && nT > 0) {
          // the k-th member of T in id order
          const uint64_t z = splitmix64_at(m.rand_seed, r);
          const uint32_t kth = (uint32_t)(((z >> 32) * (uint64_t)nT) >> 32);
          if (tid == 0) sh.pick = ~0u;
          uint32_t seen = 0;
          for (int32_t base = 0; base < n_inst; base += NT) {
            const int32_t i = base + tid;
            bool inT = false;
            if (i < n_inst) {
              const InstState st = a.inst[i];
              if (eligible(m, st.A1, st.S, L))
                inT = member(sa, m, (uint32_t)i, H[i], L, Lf, wmin, Z, kvc, slo).inT;
            }
            const uint64_t mm = __ballot(inT);
            if (lane == 0) sh.part[pb][wv].nT = (uint32_t)__popcll(mm);
            __syncthreads();
            uint32_t before = seen, tot = 0;
            for (int k = 0; k < nwv; ++k) {
              const uint32_t cn = sh.part[pb][k].nT;
              if (k < wv) before += cn;
              tot += cn;
            }
            pb ^= 1;
            if (seen + tot > kth) {
              if (inT && before + (uint32_t)__popcll(mm & lt_mask) == kth) sh.pick = (uint32_t)i;
              __syncthreads();
              keyT = sh.pick < (uint32_t)n_inst ? (uint64_t)sh.pick : ~0ull;
              break;
            }
            seen += tot;
          }
        }

        // Decision.  With finite arithmetic C holds the minimum-penalty
        // candidate whenever A is non-empty; the key test only keeps a
        // non-finite model from selecting an out-of-range id.
        if (keyT != ~0ull || keyF != ~0ull) {
          fl = 0;
          if (keyT != ~0ull) {
            best = (int32_t)(keyT & 0xFFFFu);
          } else {
            best = (int32_t)(keyF & 0xFFFFu);
            fl |= PS_R_FALLBACK;
          }
        }
      }
    }
    }  // !fast

    // (4) result and commit
    if (best >= 0 && best % NT == tid) {
      const uint32_t v = H[best];
      const int64_t c_tok = (int64_t)v * m.bs;
      InstState st = a.inst[best];
      if (!test_bit(dirty, (uint32_t)best) && sh.n_u < (uint32_t)kSpecBatch) {
        sh.u_id[sh.n_u] = (uint32_t)best;  // first placement on it in this launch
        sh.u_old[sh.n_u] = st;
        sh.n_u += 1u;
      }
      const Lat lt = latency(m, st, (float)(L - c_tok), (float)c_tok, L);
      if (lt.ttft > slo) fl |= PS_R_TTFT_MISS;
      a.out[r] = ps_result{best, (int32_t)v, lt.ttft, lt.tpot, fl};
      if (a.sizes) {
        a.sizes[3 * (size_t)r] = nA;
        a.sizes[3 * (size_t)r + 1] = nC;
        a.sizes[3 * (size_t)r + 2] = nT;
      }
      st.Q += 1;
      st.A1 += 1;
      st.P += L - c_tok;
      st.S += L;
      st.seg = segment_of(m, st.A1);
      a.inst[best] = st;
      a.room[best] = st.A1 <= m.b_max ? m.kv_cap - st.S : -1;
      dirty[best >> 6] |= 1ull << (best & 63);
      sh.hit = v;
      sh.count = a.t.count[best];
    } else if (best < 0 && tid == 0) {
      a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
      if (a.sizes) {
        a.sizes[3 * (size_t)r] = nA;
        a.sizes[3 * (size_t)r + 1] = nC;
        a.sizes[3 * (size_t)r + 2] = nT;
      }
    }
    if (best < 0) continue;
    __syncthreads();
    const uint32_t inst = (uint32_t)best;
    const int32_t v0 = (int32_t)sh.hit;
    const uint32_t count0 = sh.count;
    uint64_t* rows = a.t.rows + (size_t)inst * a.t.row_cap;
    uint32_t* rowpos = a.t.rowpos + (size_t)inst * a.t.slots;
    if ((int64_t)count0 + (ell - v0) <= (int64_t)a.cap) {
      // No block can be refused: all positions at once; a key claimed by
      // another position of the request (a repeat) is not a new block.
      uint64_t* tab = a.t.keys + (size_t)inst * (size_t)a.t.slots;
      uint32_t added = 0;
      for (int32_t p0 = v0; p0 < ell; p0 += NT * kSeqU) {
        uint64_t key[kSeqU];
        uint32_t bkt[kSeqU];
        Bucket bk[kSeqU];
#pragma unroll
        for (int u = 0; u < kSeqU; ++u) {
          const int32_t j = p0 + u * NT + tid;
          key[u] = j < ell ? seq_key(sh, c, j) : 0ull;
          bkt[u] = bucket_of(key[u], inst, a.t.shift);
          if (key[u] != 0ull) bk[u] = load_bucket(tab + (size_t)bkt[u] * kSlotsPerBucket);
        }
        bool won[kSeqU];
        uint32_t slot[kSeqU];
#pragma unroll
        for (int u = 0; u < kSeqU; ++u) {
          won[u] = false;
          slot[u] = 0;
          if (key[u] == 0ull) continue;
          int hit = -1, empty = -1;
#pragma unroll
          for (int s = 0; s < kSlotsPerBucket; ++s) {
            if (bk[u].k[s] == key[u]) hit = s;
            if (bk[u].k[s] == 0ull && empty < 0) empty = s;
          }
          if (hit >= 0) continue;
          if (empty >= 0) {
            uint64_t* sp = tab + (size_t)bkt[u] * kSlotsPerBucket + empty;
            const unsigned long long old = atomicCAS(reinterpret_cast<unsigned long long*>(sp), 0ull,
                                                     (unsigned long long)key[u]);
            if (old == 0ull) {
              won[u] = true;
              slot[u] = bkt[u] * kSlotsPerBucket + (uint32_t)empty;
              continue;
            }
            if (old == key[u]) continue;
          }
          won[u] = insert_key(a.t, inst, key[u], &slot[u]) == 1;
        }
        uint32_t rk[kSeqU];
#pragma unroll
        for (int u = 0; u < kSeqU; ++u) {
          const uint64_t wm = __ballot(won[u]);
          rk[u] = (uint32_t)__popcll(wm & lt_mask);
          if (lane == 0) sh.cnt[u][wv] = (uint32_t)__popcll(wm);
        }
        __syncthreads();
        uint32_t before[kSeqU], total = 0;
#pragma unroll
        for (int u = 0; u < kSeqU; ++u) {
          before[u] = total;
          for (int k = 0; k < nwv; ++k) {
            if (k < wv) before[u] += sh.cnt[u][k];
            total += sh.cnt[u][k];
          }
        }
#pragma unroll
        for (int u = 0; u < kSeqU; ++u) {
          if (!won[u]) continue;
          const uint32_t pos = count0 + added + before[u] + rk[u];
          rows[pos] = key[u];
          rowpos[slot[u]] = pos;
        }
        added += total;
        __syncthreads();  // cnt is rewritten by the next step
      }
      if (tid == 0) a.t.count[inst] = count0 + added;
    } else {
      // The cap binds: blocks enter in chain order until it is reached
      // (wave 0, position by position); past that point every absent block
      // is refused, counted by the whole workgroup.
      if (wv == 0) {
      uint32_t count = count0;
      int32_t stop = ell;
      for (int32_t base = v0; base < ell; base += 64) {
        if (count >= a.cap) {
          stop = base;
          break;
        }
        const int32_t j = base + lane;
        const bool in = j < ell;
        const uint64_t key = in ? seq_key(sh, c, j) : 0ull;
        const bool present = in && key != 0ull ? probe(a.t, inst, key) : true;
        // repeated keys inside this chunk: only the first occurrence counts
        int first = lane;
        for (int sl = 63; sl >= 0; --sl) {
          const uint64_t o = __shfl(key, sl);
          if (sl < lane && o == key) first = sl;
        }
        const bool dup = first != lane;
        const bool want = !present && !dup;
        const uint64_t wm = __ballot(want);
        const uint32_t rank = (uint32_t)__popcll(wm & lt_mask);
        const uint32_t room = a.cap > count ? a.cap - count : 0u;
        const bool ins = want && rank < room;
        if (ins) {  // new blocks join the row in chain order
          uint32_t slot = 0;
          (void)insert_key(a.t, inst, key, &slot);
          rows[count + rank] = key;
          rowpos[slot] = count + rank;
        }
        const uint64_t im = __ballot(ins);
        const uint64_t dup_drop = __ballot(!present && dup && !((im >> first) & 1ull));
        const uint32_t nins = (uint32_t)__popcll(im);
        count += nins;
        drop += (unsigned long long)(__popcll(wm) - nins + __popcll(dup_drop));
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");  // later probes see these inserts
      }
      if (lane == 0) {
        a.t.count[inst] = count;
        sh.ring[0] = (uint32_t)stop;
        sh.ring[1] = 0u;
      }
      }
      __syncthreads();
      const int32_t stop = (int32_t)sh.ring[0];
      if (stop < ell) {
        const uint64_t* tab = a.t.keys + (size_t)inst * (size_t)a.t.slots;
        uint32_t absent = 0;
        for (int32_t p0 = stop; p0 < ell; p0 += NT * kSeqU) {
          uint64_t key[kSeqU];
          Bucket bk[kSeqU];
#pragma unroll
          for (int u = 0; u < kSeqU; ++u) {
            const int32_t j = p0 + u * NT + tid;
            key[u] = j < ell ? seq_key(sh, c, j) : 0ull;
            if (key[u] != 0ull)
              bk[u] = load_bucket(tab + (size_t)bucket_of(key[u], inst, a.t.shift) * kSlotsPerBucket);
          }
#pragma unroll
          for (int u = 0; u < kSeqU; ++u) {
            if (key[u] == 0ull) continue;
            bool f = false, e = false;
#pragma unroll
            for (int sl = 0; sl < kSlotsPerBucket; ++sl) {
              f |= bk[u].k[sl] == key[u];
              e |= bk[u].k[sl] == 0ull;
            }
            if (!f && !e) f = probe(a.t, inst, key[u]);
            absent += f ? 0u : 1u;
          }
        }
        absent = wave_sum_u32(absent);
        if (lane == 0 && absent) atomicAdd(&sh.ring[1], absent);
        __syncthreads();
        if (tid == 0) drop += sh.ring[1];
      }
    }
  }
  if (tid == 0 && drop) atomicAdd(a.dropped, drop);
  if (tid == 0 && a.stats && (sh.n_fast | sh.n_full)) {
    atomicAdd(a.stats, (unsigned long long)sh.n_fast);
    atomicAdd(a.stats + 1, (unsigned long long)sh.n_full);
  }
}

// ------------------------------------------------ speculative batch scoring
// The kSpecTop least keys a thread has seen, ascending (keys are distinct:
// each ends in its instance id).
struct SpecTop {
  uint64_t k[kSpecTop];
  uint32_t w[kSpecTop];
};

__device__ __forceinline__ void spec_push(SpecTop& t, uint64_t key, uint32_t w) {
  if (!(key < t.k[kSpecTop - 1])) return;
  t.k[kSpecTop - 1] = key;
  t.w[kSpecTop - 1] = w;
#pragma unroll
  for (int j = kSpecTop - 1; j > 0; --j) {
    if (t.k[j] < t.k[j - 1]) {
      const uint64_t x = t.k[j];
      t.k[j] = t.k[j - 1];
      t.k[j - 1] = x;
      const uint32_t y = t.w[j];
      t.w[j] = t.w[j - 1];
      t.w[j - 1] = y;
    }
  }
}

struct SpecShared {
  uint64_t tk[kSpecTop][kSeqMaxThreads];  // each thread's candidates of T, then of C
  uint64_t fk[kSpecTop][kSeqMaxThreads];
  uint32_t tw[kSpecTop][kSeqMaxThreads];
  uint32_t fw[kSpecTop][kSeqMaxThreads];
  uint64_t red[2][2][kSeqWaves];          // per-wave minima of a merge round (alternating)
  uint32_t cnt[4][kSeqWaves];             // |A|, W_min, |C|, |T| partials
  uint32_t stop[2][2];                    // [round parity][list]: a thread that kept only part
                                          // of its members ran out (read in the next round)
};

// One workgroup per request of a batch: Algorithm 1's sets against the
// state at the batch's start (hits from the batch's hits pass), exactly as
// the scheduler evaluates them (same device functions, same fp32 values),
// without a decision: |A|, |C|, |T|, W_min and the first kSpecList members
// of T by the selector's key and of C by the fallback key.  Each thread
// keeps its kSpecTop least keys; the merge takes the least head over the
// threads, one per round, and stops after taking the last kept key of a
// thread that saw more members than it kept (its next member is unknown),
// so every list is the exact start of the ordered set.  Keyed selectors
// only (not Random, not H-C-Q).
__global__ __launch_bounds__(kSeqMaxThreads) void spec_kernel(SeqArgs a, SpecRec* out) {
  __shared__ SpecShared sh;
  const int tid = threadIdx.x, NT = blockDim.x;
  const int lane = tid & 63, wv = tid >> 6, nwv = NT >> 6;
  const int32_t n_inst = a.n_inst;
  const int32_t r = a.r0 + (int32_t)blockIdx.x;
  const ps_req q = a.reqs[r];
  if (!req_valid(q, a.pool_len)) return;  // the scheduler rejects it without a look here
  const DevModel& m = *a.model;
  const int64_t L = ((int64_t)q.pre_len + q.tail_len) * m.bs;
  const float Lf = (float)L;
  const float Z = recompute_raw(m, Lf, Lf);
  const float slo = fmaxf(m.ttft_floor, t_prefill(m, Lf, 0.0f));
  const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
  const uint32_t* H = a.hits + (size_t)blockIdx.x * (size_t)n_inst;
  SpecRec* o = out + blockIdx.x;

  // |A| and W_min
  uint32_t al = 0, wl = 0x7F800000u;
  for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
    InstState st[kSeqB];
    uint32_t hv[kSeqB];
#pragma unroll
    for (int u = 0; u < kSeqB; ++u) {
      const int32_t i = base + u * NT + tid;
      if (i < n_inst) {
        st[u] = a.inst[i];
        hv[u] = H[i];
      }
    }
#pragma unroll
    for (int u = 0; u < kSeqB; ++u) {
      if (base + u * NT + tid >= n_inst || !eligible(m, st[u].A1, st[u].S, L)) continue;
      ++al;
      const uint32_t wb =
          __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)hv[u] * m.bs), Lf)));
      wl = wb < wl ? wb : wl;
    }
  }
  al = wave_sum_u32(al);
  wl = wave_min_u32(wl);
  if (lane == 0) {
    sh.cnt[0][wv] = al;
    sh.cnt[1][wv] = wl;
  }
  if (tid < 4) sh.stop[tid >> 1][tid & 1] = 0u;
  __syncthreads();
  uint32_t nA = 0, wmin_bits = 0x7F800000u;
  for (int k = 0; k < nwv; ++k) {
    nA += sh.cnt[0][k];
    wmin_bits = sh.cnt[1][k] < wmin_bits ? sh.cnt[1][k] : wmin_bits;
  }
  const float wmin = __uint_as_float(wmin_bits);

  // members of C and T with their keys
  SpecTop tt, ff;
#pragma unroll
  for (int j = 0; j < kSpecTop; ++j) {
    tt.k[j] = ff.k[j] = ~0ull;
    tt.w[j] = ff.w[j] = 0u;
  }
  uint32_t cC = 0, cT = 0;
  if (nA > 0) {
    for (int32_t base = 0; base < n_inst; base += kSeqB * NT) {
      InstState st[kSeqB];
      uint32_t hv[kSeqB];
#pragma unroll
      for (int u = 0; u < kSeqB; ++u) {
        const int32_t i = base + u * NT + tid;
        if (i < n_inst) {
          st[u] = a.inst[i];
          hv[u] = H[i];
        }
      }
#pragma unroll
      for (int u = 0; u < kSeqB; ++u) {
        const int32_t i = base + u * NT + tid;
        if (i >= n_inst || !eligible(m, st[u].A1, st[u].S, L)) continue;
        const InstState su = st[u];
        const Member mb = member_with(m, [&]() { return su; }, hv[u], L, Lf, wmin, Z, kvc, slo);
        if (!mb.inC) continue;
        const uint32_t wb =
            __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)hv[u] * m.bs), Lf)));
        ++cC;
        const uint64_t lm = (uint64_t)(mb.st.P + mb.n_tok) * (uint64_t)mb.st.A1;
        const uint64_t kf =
            (m.flags & PS_F_FALLBACK_DCQ) ? dcq_key(mb.st, hv[u], (uint32_t)i) : ((lm << 16) | (uint32_t)i);
        spec_push(ff, kf, wb);
        if (!mb.inT) continue;
        ++cT;
        spec_push(tt, select_key(m.sel, mb.st, hv[u], (uint32_t)i, lm), wb);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kSpecTop; ++j) {
    sh.tk[j][tid] = tt.k[j];
    sh.tw[j][tid] = tt.w[j];
    sh.fk[j][tid] = ff.k[j];
    sh.fw[j][tid] = ff.w[j];
  }
  {
    const uint32_t sc = wave_sum_u32(cC), st = wave_sum_u32(cT);
    if (lane == 0) {
      sh.cnt[2][wv] = sc;
      sh.cnt[3][wv] = st;
    }
  }
  __syncthreads();
  uint32_t nC = 0, nT = 0;
  for (int k = 0; k < nwv; ++k) {
    nC += sh.cnt[2][k];
    nT += sh.cnt[3][k];
  }

  // merge: the least heads, one per round
  const int lenT = cT < (uint32_t)kSpecTop ? (int)cT : kSpecTop;
  const int lenF = cC < (uint32_t)kSpecTop ? (int)cC : kSpecTop;
  const bool cutT = cT > (uint32_t)kSpecTop, cutF = cC > (uint32_t)kSpecTop;
  int pT = 0, pF = 0, pb = 0;
  uint32_t nLT = 0, nLF = 0;
  bool doneT = nT == 0u, doneF = nC == 0u;
  for (int round = 0; round < kSpecList && !(doneT && doneF); ++round) {
    const uint64_t hT = (!doneT && pT < lenT) ? sh.tk[pT][tid] : ~0ull;
    const uint64_t hF = (!doneF && pF < lenF) ? sh.fk[pF][tid] : ~0ull;
    const uint64_t mT = wave_min_u64(hT), mF = wave_min_u64(hF);
    if (lane == 0) {
      sh.red[pb][0][wv] = mT;
      sh.red[pb][1][wv] = mF;
    }
    __syncthreads();
    uint64_t gT = ~0ull, gF = ~0ull;
    for (int k = 0; k < nwv; ++k) {
      gT = sh.red[pb][0][k] < gT ? sh.red[pb][0][k] : gT;
      gF = sh.red[pb][1][k] < gF ? sh.red[pb][1][k] : gF;
    }
    pb ^= 1;
    // written in the previous round (each round writes the slot the next
    // one reads, after a barrier that every reader of the slot has passed)
    if (sh.stop[round & 1][0]) doneT = true;
    if (sh.stop[round & 1][1]) doneF = true;
    if (!doneT) {
      if (gT == ~0ull) {
        doneT = true;
      } else {
        if (hT == gT) {
          o->lt[nLT] = SpecEntry{gT, sh.tw[pT][tid], 0u};
          if (++pT == lenT && cutT) sh.stop[(round + 1) & 1][0] = 1u;
        }
        ++nLT;
      }
    }
    if (!doneF) {
      if (gF == ~0ull) {
        doneF = true;
      } else {
        if (hF == gF) {
          o->lf[nLF] = SpecEntry{gF, sh.fw[pF][tid], 0u};
          if (++pF == lenF && cutF) sh.stop[(round + 1) & 1][1] = 1u;
        }
        ++nLF;
      }
    }
  }
  if (tid == 0) {
    o->nA = nA;
    o->nC = nC;
    o->nT = nT;
    o->wmin = wmin_bits;
    o->nLT = nLT;
    o->nLF = nLF;
  }
}

}  // namespace

hipError_t ps_launch_spec(const SeqArgs& a, SpecRec* out, hipStream_t s) {
  if (a.r1 <= a.r0) return hipSuccess;
  hipLaunchKernelGGL(spec_kernel, dim3(a.r1 - a.r0), dim3(kSeqMaxThreads), 0, s, a, out);
  return hipGetLastError();
}

size_t ps_seq_lds_bytes(int32_t n_inst) {
  const size_t nw = ((size_t)n_inst + 63) / 64;
  return sizeof(SeqShared) + nw * sizeof(uint64_t);
}

hipError_t ps_launch_seq(const SeqArgs& a, int threads, hipStream_t s) {
  if (a.r1 <= a.r0) return hipSuccess;
  if (threads < 64 || threads > kSeqMaxThreads || threads % 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(seq_kernel, dim3(1), dim3(threads), ps_seq_lds_bytes(a.n_inst), s, a);
  return hipGetLastError();
}
