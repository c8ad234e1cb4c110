// HIP kernels of the window scorer for gfx950 (CDNA4, wave64).
//
//   build_kernel      - per-instance open-addressing tables from the CSR block
//                       lists (64-bit atomicCAS inserts).
//   score_kernel      - the fused hot path, one wave per request:
//                         (1) longest cached prefix on every capacity-eligible
//                             instance.  One prefix-index lookup of the first
//                             block gives the instances that hold it; every
//                             other eligible instance has hit 0.  Up to 64
//                             holders are walked on their own tables (octets of
//                             lanes over chain positions, the first absent
//                             block from a ballot); more holders are walked
//                             together through the index, position by
//                             position, with LDS bitmaps of the live set.
//                             The chain head is staged in LDS.
//                         (2) the latency model (Eq. 7 + C, C^2 terms; Eq. 8
//                             per segment with its EMA factor; Eq. 10; Eq. 4),
//                         (3) capacity, recomputation (Eq. 9) and TPOT filters:
//                             all hit-0 instances share one penalty, so that
//                             class is evaluated only if it passes Eq. 9,
//                         (4) the packed D-C-Q and LMetric keys, reduced with
//                             DPP wave minima.
//   probe_all_kernel  - diagnostic: the hit of every request on every
//                       instance by direct probing of the per-instance tables
//                       (breadth probe of the first block, then deep walks;
//                       one lane per probe, a whole bucket per lane).
//   commit_kernel     - ordered placement of decisions, one wave per instance.
//
// The path does no dense contraction, so it uses no MFMA.

#include "ps_common.h"

namespace {

// ------------------------------------------------------------------ kernels
__global__ void build_kernel(BuildArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < a.n_blk; k += stride) {
    int32_t lo = 0, hi = a.n_inst;  // last row with blk_off[row] <= k
    while (hi - lo > 1) {
      const int32_t mid = (lo + hi) >> 1;
      if (a.blk_off[mid] <= k) lo = mid;
      else hi = mid;
    }
    uint32_t slot = 0;
    const int r = insert_key(a.t, (uint32_t)lo, a.blk[k], &slot);
    // One counter update per wave when its lanes share the instance (a
    // list is contiguous), instead of one contended atomic per key.
    const int lane = threadIdx.x & 63;
    const uint64_t act = __ballot(1);
    const int leader = __builtin_ctzll(act);
    const int32_t lo0 = __shfl(lo, leader);
    if (__ballot(lo == lo0) == act) {
      const uint64_t wm = __ballot(r == 1);
      if (lane == leader && wm) atomicAdd(&a.t.count[lo0], (uint32_t)__popcll(wm));
    } else if (r == 1) {
      atomicAdd(&a.t.count[lo], 1u);
    }
    if (r < 0) atomicAdd(a.full, 1ull);
    a.won[k] = r == 1 ? 1u : 0u;
    a.slot_of[k] = slot;
  }
}

// Rows: the entries that inserted their key, in list order, become the
// instance's row; rank is the global exclusive scan of `won`.
__global__ void row_kernel(BuildArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < a.n_blk; k += stride) {
    if (!a.won[k]) continue;
    int32_t lo = 0, hi = a.n_inst;
    while (hi - lo > 1) {
      const int32_t mid = (lo + hi) >> 1;
      if (a.blk_off[mid] <= k) lo = mid;
      else hi = mid;
    }
    const uint32_t pos = a.rank[k] - a.rank[a.blk_off[lo]];
    a.t.rows[(size_t)lo * a.t.row_cap + pos] = a.blk[k];
    a.t.rowpos[(size_t)lo * a.t.slots + a.slot_of[k]] = pos;
  }
}

// Hit of every request on every instance by direct probing, one wave per
// request.  Lane l probes the first block on instance base + 64 r + l (BR x
// 64 instances per step, a whole 64-byte bucket per lane), then each
// instance that holds it is walked with DR x 64 positions per step.
template <int BR, int DR>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4))) void probe_all_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  const int lane = threadIdx.x;
  const int32_t n_inst = a.n_inst;
  // With an order: the order's chunks of kOrderChunk requests are dealt to
  // the XCDs in turn (workgroup b runs on XCD b % kXcds), and each XCD takes
  // its chunks in order.  Otherwise array order.
  const int32_t x = (int32_t)(blockIdx.x % kXcds);
  const int32_t gx = (int32_t)(gridDim.x / kXcds);
  for (int32_t i = (int32_t)(blockIdx.x / kXcds), w0 = (int32_t)blockIdx.x;; i += gx, w0 += gridDim.x) {
    const int64_t w = a.req_order ? ((int64_t)x + (int64_t)kXcds * (i / kOrderChunk)) * kOrderChunk +
                                        i % kOrderChunk
                                  : (int64_t)w0;
    if (w >= a.n_req) break;
    const int32_t r = a.req_order ? a.req_order[w] : w;
    const ps_req q = a.reqs[r];
    if (!req_valid(q, a.pool_len)) {
      for (int32_t k = lane; k < n_inst; k += 64) a.hits_out[(size_t)r * n_inst + k] = 0xFFFFFFFFu;
      continue;
    }
    const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
    const int32_t ell = c.len;
    const int32_t nst = ell < kStage ? ell : kStage;
    __syncthreads();
    for (int32_t j = lane; j < nst; j += 64) stage[j] = chain_global(c, j);
    __syncthreads();
    const uint64_t k0 = ell > 0 ? stage[0] : 0ull;
    for (int32_t base = 0; base < n_inst; base += 64 * BR) {
      Bucket v[BR];
      uint32_t bkt[BR];
#pragma unroll
      for (int rr = 0; rr < BR; ++rr) {
        const uint32_t i = (uint32_t)(base + rr * 64 + lane);
        bkt[rr] = bucket_of(k0, i, a.t.shift);
        v[rr] = Bucket{};
        if ((int32_t)i < n_inst && k0 != 0ull)
          v[rr] = load_bucket(table_of(a.t, i) + (size_t)bkt[rr] * kSlotsPerBucket);
      }
#pragma unroll
      for (int rr = 0; rr < BR; ++rr) {
        const int32_t b0 = base + rr * 64;
        if (b0 >= n_inst) break;
        const uint32_t i = (uint32_t)(b0 + lane);
        uint32_t st = (int32_t)i < n_inst ? lane_status(v[rr], k0) : 0u;
        if (st == 2u) st = lane_resolve(a.t, table_of(a.t, i), bkt[rr], k0) ? 1u : 0u;
        uint32_t h = st == 1u ? 1u : 0u;
        uint64_t deep = ell > 1 ? __ballot(st == 1u) : 0ull;
        while (deep) {
          const int k = __builtin_ctzll(deep);
          deep &= deep - 1;
          const uint32_t hk = lane_walk<true, DR>(a.t, (uint32_t)(b0 + k), c, stage, 1, lane);
          if (lane == k) h = hk;
        }
        if ((int32_t)i < n_inst) a.hits_out[(size_t)r * n_inst + i] = h;
      }
    }
  }
}

// Counting sort of the requests for the exhaustive probe: by descending
// chain length in bins of 256 blocks, so that the longest walks start first
// and the launch does not end on a few long walks begun late, and within a
// length bin by a hash of the shared segment, so that requests of one
// session sit together and share the L2 of one XCD.  Within a bin the
// order is arbitrary: every request's hits go to its own row.
__device__ __forceinline__ uint32_t order_bin(const ps_req& q, int64_t pool_len) {
  if (!req_valid(q, pool_len)) return kOrderAll - 1;
  const int64_t b = ((int64_t)q.pre_len + q.tail_len) >> kOrderShift;
  const uint32_t lb = (uint32_t)(kOrderLenBins - 1) - (uint32_t)(b < kOrderLenBins - 1 ? b : kOrderLenBins - 1);
  const uint32_t hb = (uint32_t)(((uint64_t)q.pre_off * 0x9E3779B97F4A7C15ull) >> 56);
  return lb * kOrderHashBins + hb;
}

__global__ void order_clear_kernel(uint32_t* bins) {
  for (int32_t i = threadIdx.x; i < kOrderAll; i += blockDim.x) bins[i] = 0u;
}

// Lanes of a wave with the same bin add to it once (one lane, the count of
// them): a popular session would otherwise serialise thousands of atomics on
// one bin.  Returns, in every active lane, the bin's old value plus the
// lane's rank among those lanes.
__device__ __forceinline__ uint32_t wave_bin_add(uint32_t* bins, uint32_t bin, bool act) {
  const int lane = threadIdx.x & 63;
  // each lane's leader (the lowest lane with its bin), rank and, in the
  // leader, the count: ballots only
  uint64_t todo = __ballot(act);
  int leader = lane;
  uint32_t rank = 0u, cnt = 0u;
  while (todo) {
    const int src = __builtin_ctzll(todo);
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)bin, src);
    const uint64_t same = __ballot(act && bin == b);
    todo &= ~same;
    if (act && bin == b) {
      leader = src;
      rank = (uint32_t)__popcll(same & ((1ull << lane) - 1ull));
      cnt = (uint32_t)__popcll(same);
    }
  }
  // then all leaders' atomics at once
  uint32_t base = 0u;
  if (act && leader == lane) base = atomicAdd(&bins[bin], cnt);
  return (uint32_t)__shfl((int)base, leader) + rank;
}

__global__ void order_count_kernel(const ps_req* reqs, int32_t n, int64_t pool_len, uint32_t* bins) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  const bool act = i < n;
  (void)wave_bin_add(bins, act ? order_bin(reqs[i], pool_len) : 0u, act);
}

// Exclusive prefix sum of the bin counts in place (one workgroup of
// 1,024 threads): each bin's first position in the order.
__global__ __launch_bounds__(1024) void order_scan_kernel(uint32_t* bins) {
  constexpr int E = kOrderAll / 1024;  // bins per thread
  __shared__ uint32_t wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  uint32_t v[E], tot = 0u;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    v[e] = bins[tid * E + e];
    tot += v[e];
  }
  const uint32_t ex = wave_exclusive_sum(tot, lane);
  if (lane == 63) wsum[wv] = ex + tot;
  __syncthreads();
  if (wv == 0) {
    const uint32_t t = lane < 16 ? wsum[lane] : 0u;
    const uint32_t te = wave_exclusive_sum(t, lane);
    if (lane < 16) wsum[lane] = te;
  }
  __syncthreads();
  uint32_t run = wsum[wv] + ex;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int32_t k = tid * E + e;
    bins[k] = run;
    run += v[e];
  }
}

__global__ void order_place_kernel(const ps_req* reqs, int32_t n, int64_t pool_len, uint32_t* bins,
                                   int32_t* order) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  const bool act = i < n;
  const uint32_t pos = wave_bin_add(bins, act ? order_bin(reqs[i], pool_len) : 0u, act);
  if (act) order[pos] = i;
}

// Zero-hit admission threshold of the instance at key position k: the
// longest chain (blocks) it admits with no cached prefix, i.e. capacity-
// eligible and, unless the TPOT test is off, predicted TPOT below the
// target.  With a monotone model both tests hold for every shorter chain
// too, so a binary search over the length finds the boundary with the same
// fp32 evaluation the scoring kernel makes; -1 when not even an empty
// chain is admitted.  lm1 = the maximum over each 64-entry chunk.
__global__ __launch_bounds__(64) void lmax_kernel(const InstState* inst_key, const uint32_t* order0,
                                                  const DevModel* mp, int32_t n, int4* lm,
                                                  int32_t* lm1, uint4* csum) {
  const DevModel& m = *mp;
  const int32_t k = blockIdx.x * 64 + threadIdx.x;
  int32_t best = -1;
  uint32_t tb = 0xFFFFFFFFu, ti = 0xFFFFFFFFu;  // order-preserving bits (sortable_bits)
  uint64_t rm1 = 0ull;                           // room + 1
  if (k < n) {
    const InstState st = inst_key[k];
    // the chunk summary for scans of a class with c > 0 (every member's
    // TPOT is at least its t_iter at L = 0 plus the class's interference
    // when A1 > 1, under a monotone model)
    const uint32_t t0 = sortable_bits(t_iter_of(m, st, 0));
    if (st.A1 > 1) tb = t0;
    else ti = t0;
    const int64_t room = st.A1 <= m.b_max ? m.kv_cap - st.S : -1;
    rm1 = room >= 0 ? (uint64_t)(room + 1) : 0ull;
    auto admits = [&](int32_t ell) {
      const int64_t L = (int64_t)ell * m.bs;
      if (!eligible(m, st.A1, st.S, L)) return false;
      if (m.flags & PS_F_NO_TPOT_FILTER) return true;
      return latency(m, st, (float)L, 0.0f, L).tpot < m.tau;
    };
    if (admits(0)) {
      int32_t lo = 0, hi = PS_MAX_CHAIN + 1;  // admits(lo); hi fails or lies past the range
      while (hi - lo > 1) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (admits(mid)) lo = mid;
        else hi = mid;
      }
      best = lo;
    }
    lm[k] = make_int4(best, (int)order0[k], st.D, st.Q);
  }
  const uint64_t mx = ~wave_min_u64(~(uint64_t)(uint32_t)(best + 1));
  const uint32_t tbm = wave_min_u32(tb), tim = wave_min_u32(ti);
  const uint64_t rmx = ~wave_min_u64(~rm1) - 1ull;
  auto unsort = [](uint32_t b) {  // inverse of sortable_bits (all ones: +inf, no member)
    return b == 0xFFFFFFFFu ? 0x7F800000u : ((b & 0x80000000u) ? (b & 0x7FFFFFFFu) : ~b);
  };
  if (threadIdx.x == 0) {
    lm1[blockIdx.x] = (int32_t)mx - 1;
    csum[blockIdx.x] = make_uint4(unsort(tbm), unsort(tim), (uint32_t)rmx, (uint32_t)(rmx >> 32));
  }
}

// Hits of the live holders (the bits of bmA, nalive of them, all holding
// the chain's first p blocks), walked together through the prefix index:
// eight positions per batched lookup; each position's holders (a list, or
// a bitmap for popular hashes) intersect the live set, and an instance that
// drops out at position pos gets put(id, pos); a single survivor continues
// on its own row, and survivors of the whole chain get put(id, ell).  bmN
// must be clear; both bitmaps are clear on return.  Wave-uniform arguments.
// PF: on pools of at most 4,096 instances (one bitmap word per lane) the
// holder bitmaps of a batch's popular positions are loaded together, before
// the batch is applied in order.  RW, RU0: positions per lane of the
// single-holder row walk's steps (run_walk).  BULK (pools of at most 4,096
// instances): when a listed position drops many holders at once, their
// put calls go word by word with the lanes over the word's bits (one
// coalesced round of stores per word) rather than bit by bit per lane.
template <bool STAGED, bool PF, int RW = kWalkU, int RU0 = 4, bool BULK = false, class Put>
__device__ __forceinline__ void index_walk(const ScoreArgs& a, const ChainRef& c,
                                           const uint64_t* stage, uint64_t* bmA, uint64_t* bmN,
                                           int32_t nw, uint32_t nalive, int32_t p, Put put,
                                           int lane, int g, int s) {
  const int32_t ell = c.len;
  const bool pf = PF && nw <= 64;
  while (p < ell && nalive > 0) {
    if (nalive == 1) {  // a single live holder: walk its own table
      uint32_t who = 0;
      for (int32_t w0 = 0; w0 < nw; w0 += 64) {
        const int32_t w = w0 + lane;
        const uint64_t word = w < nw ? bmA[w] : 0ull;
        const uint64_t any = __ballot(word != 0ull);
        if (any) {
          const int ln = __builtin_ctzll(any);
          const uint64_t wd = __shfl(word, ln);
          who = (uint32_t)((w0 + ln) * 64 + __builtin_ctzll(wd));
          break;
        }
      }
      const uint32_t hk = run_walk<STAGED, RW, RU0>(a.t, who, c, stage, p, g, s);
      if (lane == 0) {
        put(who, hk);
        bmA[who >> 6] = 0ull;
      }
      nalive = 0;
      __syncthreads();
      break;
    }
    const int32_t jq = p + g;
    const uint64_t kq =
      jq < ell ? ((STAGED && jq < kStage) ? stage[jq] : chain_global(c, jq)) : 0ull;
    const IdxHit hq = index_lookup(a.x, kq, jq < ell, g, s);
    uint64_t pw[8];
    if (PF) {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const bool f = __shfl(hq.found ? 1 : 0, 8 * t) != 0;
        const uint32_t off = __shfl(hq.off, 8 * t), cnt = __shfl(hq.cnt, 8 * t);
        pw[t] = pf && f && cnt > kPopular && lane < nw ? a.x.bitmaps[(size_t)off * a.x.nw + lane] : 0ull;
      }
    }
    int32_t used = 0;
    constexpr int kUnroll = PF ? 8 : 1;  // (pw stays in registers)
#pragma unroll kUnroll
    for (int t = 0; t < 8; ++t) {
      const int32_t pos = p + t;
      if (pos >= ell || nalive <= 1) break;
      const bool f = __shfl(hq.found ? 1 : 0, 8 * t) != 0;
      const uint32_t off = __shfl(hq.off, 8 * t), cnt = __shfl(hq.cnt, 8 * t);
      if (f && cnt > kPopular) {  // live &= holder bitmap, lane-owned words
        const uint64_t* bm = a.x.bitmaps + (size_t)off * a.x.nw;
        uint32_t live = 0;
        if (BULK && nw <= 64) {
          const uint64_t aw = lane < nw ? bmA[lane] : 0ull;
          const uint64_t nwd = aw & (lane < nw ? (pf ? pw[t] : bm[lane]) : 0ull);
          const uint64_t d = aw & ~nwd;
          if (__ballot(__popcll(d) > 4u)) {
            for (int32_t w = 0; w < nw; ++w) {
              const uint64_t dw = (uint64_t)lane_value64((int64_t)d, w);
              if ((dw >> lane) & 1ull) put((uint32_t)(w * 64 + lane), (uint32_t)pos);
            }
          } else {
            uint64_t dd = d;
            while (dd) {
              const int b = __builtin_ctzll(dd);
              dd &= dd - 1;
              put((uint32_t)(lane * 64 + b), (uint32_t)pos);
            }
          }
          if (lane < nw) bmA[lane] = nwd;
          live = (uint32_t)__popcll(nwd);
        } else {
          for (int32_t w = lane; w < nw; w += 64) {
            const uint64_t aw = bmA[w];
            const uint64_t nwd = aw & (pf ? pw[t] : bm[w]);
            uint64_t d = aw & ~nwd;
            while (d) {
              const int b = __builtin_ctzll(d);
              d &= d - 1;
              put((uint32_t)(w * 64 + b), (uint32_t)pos);
            }
            bmA[w] = nwd;
            live += (uint32_t)__popcll(nwd);
          }
        }
        nalive = wave_sum_u32(live);
        used = t + 1;
        continue;
      }
      if (f) {
        for (uint32_t t0 = 0; t0 < cnt; t0 += 64) {
          const uint32_t tt = t0 + lane;
          if (tt < cnt) {
            const uint32_t id = a.x.holders[off + tt];
            if (test_bit(bmA, id))
              atomicOr(reinterpret_cast<unsigned long long*>(&bmN[id >> 6]), 1ull << (id & 63));
          }
        }
      }
      __syncthreads();
      uint32_t live = 0;
      if (BULK && nw <= 64) {  // word `lane`; many leaving holders: lanes over each word's bits
        const uint64_t aw = lane < nw ? bmA[lane] : 0ull, nwd = lane < nw ? bmN[lane] : 0ull;
        uint64_t d = aw & ~nwd;
        if (__ballot(__popcll(d) > 4u)) {
          for (int32_t w = 0; w < nw; ++w) {
            const uint64_t dw = (uint64_t)lane_value64((int64_t)d, w);
            if ((dw >> lane) & 1ull) put((uint32_t)(w * 64 + lane), (uint32_t)pos);
          }
        } else {
          while (d) {
            const int b = __builtin_ctzll(d);
            d &= d - 1;
            put((uint32_t)(lane * 64 + b), (uint32_t)pos);
          }
        }
        if (lane < nw) {
          bmA[lane] = nwd;
          bmN[lane] = 0ull;
        }
        live = (uint32_t)__popcll(nwd);
      } else {
        for (int32_t w = lane; w < nw; w += 64) {
          const uint64_t aw = bmA[w], nwd = bmN[w];
          uint64_t d = aw & ~nwd;
          while (d) {
            const int b = __builtin_ctzll(d);
            d &= d - 1;
            put((uint32_t)(w * 64 + b), (uint32_t)pos);
          }
          bmA[w] = nwd;
          bmN[w] = 0ull;
          live += (uint32_t)__popcll(nwd);
        }
      }
      __syncthreads();
      nalive = wave_sum_u32(live);
      used = t + 1;
    }
    p += used;
  }
  if (nalive > 0) {  // survived to the end of the chain
    for (int32_t w = lane; w < nw; w += 64) {
      uint64_t d = bmA[w];
      while (d) {
        const int b = __builtin_ctzll(d);
        d &= d - 1;
        put((uint32_t)(w * 64 + b), (uint32_t)ell);
      }
      bmA[w] = 0ull;
    }
  }
  __syncthreads();
}

// Slot of a request's prefix group.  Linear probing over the window's
// group table; a slot whose key belongs to an older window is empty and is
// claimed with a 64-bit compare-and-swap.  Keys of the current window never
// change once written, so a plain read that shows one is exact, and a stale
// read only makes the compare-and-swap fail, whose result then decides.
// *leader = 1 for the request whose swap claimed the slot.
__device__ int32_t group_claim(const GroupTab& G, int64_t pre_off, int* leader) {
  const unsigned long long key =
      ((unsigned long long)G.gen << kGroupGenShift) | (unsigned long long)(pre_off + 1);
  uint32_t b = (uint32_t)(((uint64_t)(pre_off + 1) * 0x9E3779B97F4A7C15ull) >> 32) & G.mask;
  *leader = 0;
  for (uint32_t step = 0; step <= G.mask; ++step, b = (b + 1) & G.mask) {
    const unsigned long long v = G.keys[b];
    if (v == key) return (int32_t)b;
    if ((v >> kGroupGenShift) == G.gen) continue;  // another group of this window
    const unsigned long long old = atomicCAS(&G.keys[b], v, key);
    if (old == v) {
      *leader = 1;
      return (int32_t)b;
    }
    if (old == key) return (int32_t)b;
    // otherwise claimed for another group of this window meanwhile
  }
  return -1;  // table full (not reached: it holds at least twice the requests)
}

// Single-thread lookup in the prefix index: the 8 entries of the key's
// first bucket are read together (IdxBucket, 8 x {key, off | cnt << 32}),
// then searched (index_search, which goes on to the next buckets while a
// bucket is full without the key).  {off, cnt} of the key's entry; cnt 0
// when it is absent.
struct IdxBucket {
  ulonglong2 v0, v1, v2, v3, v4, v5, v6, v7;
};

__device__ __forceinline__ IdxBucket index_bucket(const GIndex& x, uint32_t b) {
  static_assert(sizeof(IdxEntry) == 16 && kSlotsPerBucket == 8, "a bucket is 8 x 16 bytes");
  const ulonglong2* e = reinterpret_cast<const ulonglong2*>(x.ent + (size_t)b * kSlotsPerBucket);
  return IdxBucket{e[0], e[1], e[2], e[3], e[4], e[5], e[6], e[7]};
}

__device__ __forceinline__ uint2 index_search(const GIndex& x, uint64_t key, uint32_t b,
                                              const IdxBucket& bk) {
  if (key == 0ull) return make_uint2(0u, 0u);
  for (const ulonglong2 v : {bk.v0, bk.v1, bk.v2, bk.v3, bk.v4, bk.v5, bk.v6, bk.v7}) {
    if (v.x == key) return make_uint2((uint32_t)v.y, (uint32_t)(v.y >> 32));
    if (v.x == 0ull) return make_uint2(0u, 0u);
  }
  // a full bucket without the key: the next buckets, one entry at a time
  for (uint32_t step = 1; step <= x.bmask; ++step) {
    b = (b + 1) & x.bmask;
    for (int t = 0; t < kSlotsPerBucket; ++t) {
      const IdxEntry e = x.ent[(size_t)b * kSlotsPerBucket + t];
      if (e.key == key) return make_uint2(e.off, e.cnt);
      if (e.key == 0ull) return make_uint2(0u, 0u);
    }
  }
  return make_uint2(0u, 0u);
}

// Prefix groups, pass 1 (one thread per request; the grid covers every
// request once): the slot of every request's group and the group's longest
// segment (a 64-bit maximum over generation-tagged lengths, so no slot
// needs clearing between windows).  Requests of one workgroup with the
// same segment claim once (see below); each new leader goes into a list for
// the walk pass.
constexpr int kClaimBlock = 256;  // threads (requests) per workgroup of the claim pass

__global__ __launch_bounds__(kClaimBlock) void group_claim_kernel(ScoreArgs a) {
  const GroupTab& G = a.grp;
  if (blockIdx.x == 0 && threadIdx.x == 0) {  // read only by the later kernels of this window
    G.pop_ctr[0] = 0u;
    G.pop_ctr[1] = 0u;
  }
  if (blockIdx.x == 0 && threadIdx.x < 2 * kXcds)  // the next window's list lengths and longest segments
    G.lctr_next[(threadIdx.x >> 1) * kListCtrWords + (threadIdx.x & 1u)] = 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) G.lctr_next[kPopCountWord] = 0u;  // and popular count
  if (a.dlist && blockIdx.x == 0 && threadIdx.x < kDeferLists)  // the rows scorer's hand-over
    a.dcnt[threadIdx.x * kDeferStride] = 0u;
  const int32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63;
  bool want = false;
  int64_t off = -1;
  int32_t plen = 0;
  if (r < a.n_req) {
    const ps_req q = a.reqs[r];
    want = req_valid(q, a.pool_len) && q.pre_len >= kGroupMin;
    if (want) {
      off = q.pre_off;
      plen = q.pre_len;
    }
  }
  // Requests of this workgroup with the same segment meet in an LDS hash
  // table: the lowest thread claims for all of them, with their longest
  // length (a popular session would otherwise serialise its atomics on one
  // slot).
  __shared__ unsigned long long lkey[2 * kClaimBlock];
  __shared__ int32_t llen[2 * kClaimBlock], lfirst[2 * kClaimBlock], lslot[2 * kClaimBlock];
  const int tid = threadIdx.x;
  for (int i = tid; i < 2 * kClaimBlock; i += kClaimBlock) {
    lkey[i] = 0ull;
    llen[i] = 0;
    lfirst[i] = kClaimBlock;
    lslot[i] = -1;
  }
  __syncthreads();
  int h = 0;
  if (want) {
    const unsigned long long k = (unsigned long long)(off + 1);
    uint32_t b = (uint32_t)((k * 0x9E3779B97F4A7C15ull) >> 40) & (2 * kClaimBlock - 1);
    for (int step = 0; step < 2 * kClaimBlock; ++step) {  // at most kClaimBlock keys: a free entry exists
      const unsigned long long old = atomicCAS(&lkey[b], 0ull, k);
      if (old == 0ull || old == k) break;
      b = (b + 1) & (2 * kClaimBlock - 1);
    }
    h = (int)b;
    atomicMax(&llen[h], plen);
    atomicMin(&lfirst[h], tid);
  }
  __syncthreads();
  const bool first = want && lfirst[h] == tid;
  int32_t slot = -1;
  int leader = 0;
  if (first) {
    slot = group_claim(G, off, &leader);
    if (slot >= 0)
      atomicMax(&G.plen[slot],
                ((unsigned long long)G.gen << kGroupGenShift) | (unsigned long long)llen[h]);
    lslot[h] = slot;
  }
  __syncthreads();
  static_assert(2 * kGroupMaxReq <= (1 << 24) && kGroupGenShift + 24 <= 64,
                "a list entry packs a slot (24 bits) and a segment offset (40 bits)");
  // the leaders' slots into this wave's list: one atomic per wave, lists
  // dealt to waves in turn (a list holds at most lcap entries: 64 per wave
  // that writes it)
  const bool lead = first && slot >= 0 && leader;
  const uint64_t lm = __ballot(lead);
  const uint32_t x = ((uint32_t)(blockIdx.x * blockDim.x + threadIdx.x) >> 6) % (uint32_t)kXcds;
  // a bound on every group's segment length (its claims' lengths; only
  // lengths above one part's minimum matter to the walk pass)
  // (the walk pass reads the maximum over all lists, so one atomic per
  // workgroup, on its first wave's list, with the workgroup's maximum:
  // atomics on these eight lines queue at the memory side)
  const uint32_t cmax = (uint32_t)(~wave_min_u64(~(uint64_t)(uint32_t)(first && slot >= 0 ? llen[h] : 0)));
  __shared__ uint32_t wg_cmax;
  if (tid == 0) wg_cmax = 0u;
  __syncthreads();
  if (lane == 0 && cmax > (uint32_t)kGroupPartMin) atomicMax(&wg_cmax, cmax);
  __syncthreads();
  if (tid == 0 && wg_cmax) atomicMax(&G.lctr[x * kListCtrWords + 1], wg_cmax);
  if (lm) {
    uint32_t base = 0u;
    if (lane == 0) base = atomicAdd(&G.lctr[x * kListCtrWords], (uint32_t)__popcll(lm));
    base = (uint32_t)__shfl((int)base, 0);
    if (lead) {
      G.lists[(size_t)x * G.lcap + base + (uint32_t)__popcll(lm & ((1ull << lane) - 1ull))] =
          ((unsigned long long)(off + 1) << 24) | (unsigned long long)slot;
      uint2* rec = G.rec + (size_t)slot * kGroupRec;  // hits: minima of the walk's parts
      for (uint32_t t = 0; t < kGroupHold; ++t) rec[1 + t] = make_uint2(0u, 0xFFFFFFFFu);
    }
  }
  // A leader whose first block has a holder bitmap (a popular group) goes
  // into the popular pass's list (one count atomic per workgroup) and its
  // slot into the bitmap's representative word (one plain store per bitmap
  // and wave; whichever lands last represents the bitmap).  Its class word
  // says whether it was listed; the walk pass takes the others.
  if (G.pop_pass) {
    bool pop = false;
    uint32_t off0 = 0u;
    if (lead) {
      const uint64_t key0 = a.pool[off];
      const uint32_t b = bucket_of(key0, kIndexSalt, a.x.shift);
      const uint2 f = index_search(a.x, key0, b, index_bucket(a.x, b));
      off0 = f.x;
      pop = f.y > kPopular && off0 < G.rep_cap;
    }
    const uint64_t pm = __ballot(pop);
    // one count atomic per workgroup (it shares list 0's line, whose
    // atomics queue at the memory side): waves' counts in LDS
    __shared__ uint32_t pcnt[kClaimBlock / 64], pbase;
    const int wv = tid >> 6;
    if (lane == 0) pcnt[wv] = (uint32_t)__popcll(pm);
    __syncthreads();
    if (tid == 0) {
      uint32_t tot = 0u;
      for (int k = 0; k < kClaimBlock / 64; ++k) tot += pcnt[k];
      pbase = tot ? atomicAdd(&G.lctr[kPopCountWord], tot) : 0u;
    }
    __syncthreads();
    if (pm) {
      uint32_t k0 = pbase;
      for (int k = 0; k < wv; ++k) k0 += pcnt[k];
      const uint32_t k = k0 + (uint32_t)__popcll(pm & ((1ull << lane) - 1ull));
      const bool listed = pop && k < G.plist_cap;
      if (listed) G.plist[k] = make_uint2((uint32_t)slot, off0);
      if (pop)
        G.rec[(size_t)slot * kGroupRec + kGroupClsWord] =
            make_uint2(kGroupNone, listed ? off0 : kGroupUnlisted);
      // any listed group of a bitmap can represent it (the popular pass is
      // exact for every choice), so a plain store: an atomic per wave on
      // one word would queue at the memory side
      const unsigned long long tag = (kGroupGenMax - G.gen) << 32;
      uint64_t pend = __ballot(listed);
      while (pend) {
        const int src = __builtin_ctzll(pend);
        const uint32_t o = (uint32_t)__shfl((int)off0, src);
        pend &= ~__ballot(listed && off0 == o);
        if (lane == src) G.rep[o] = tag | (unsigned long long)(uint32_t)slot;
      }
    }
  }
  if (want) slot = lslot[h];
  if (r < a.n_req)
    G.slot_of[r] = want && slot >= 0 ? (uint32_t)slot | (lead ? kGroupLead : 0u) : kGroupNoSlot;
}

// The shared-hit class of a popular group (hits of its holders in hp, the
// holders in bitmap off0): H* = the most frequent hit among the holders of
// the first 64-instance word that has any; when at most kGroupHold holders
// differ from it, the record keeps them (rec[1..]) and the result is the
// class word {n_exc << 24 | H*}, else kGroupNone.  Bitmap words are read 64
// at a time (one per lane) and hits kClassChunk words at a time, all in
// flight.  The
// wave's own hit writes are read back under a workgroup-scope fence (a
// device-scope one writes back the XCD's whole L2).
template <int kClassChunk = 8>
__device__ __forceinline__ uint32_t popular_class(const ScoreArgs& a, uint2* rec,
                                                  const uint32_t* hp, uint32_t off0, int32_t nw,
                                                  int lane) {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  const uint64_t* bm = a.x.bitmaps + (size_t)off0 * a.x.nw;
  uint32_t hs = 0u, nexc = 0u;
  bool have_hs = false;
  for (int32_t wb = 0; wb < nw && nexc <= kGroupHold; wb += 64) {
    const int32_t wn = nw - wb < 64 ? nw - wb : 64;
    const uint64_t bmw = lane < wn ? bm[wb + lane] : 0ull;
    for (int32_t w0 = 0; w0 < wn && nexc <= kGroupHold; w0 += kClassChunk) {
      bool hold[kClassChunk];
      uint32_t v[kClassChunk];
#pragma unroll
      for (int u = 0; u < kClassChunk; ++u) {
        const uint64_t word = (uint64_t)lane_value64((int64_t)bmw, (w0 + u) & 63);
        hold[u] = w0 + u < wn && ((word >> lane) & 1ull) != 0ull;
        v[u] = hold[u] ? hp[(wb + w0 + u) * 64 + lane] : 0u;
      }
      if (!have_hs) {  // the mode over the first word with holders
        uint64_t wsel = 0ull;
        uint32_t vsel = 0u;
#pragma unroll
        for (int u = 0; u < kClassChunk; ++u) {
          const uint64_t word = (uint64_t)lane_value64((int64_t)bmw, (w0 + u) & 63);
          if (!wsel && w0 + u < wn && word) {
            wsel = word;
            vsel = v[u];
          }
        }
        if (wsel) {
          const bool hold0 = ((wsel >> lane) & 1ull) != 0ull;
          uint64_t rem = wsel;
          uint32_t bestc = 0u;
          while (rem) {
            const uint32_t val = (uint32_t)__builtin_amdgcn_readlane((int)vsel, __builtin_ctzll(rem));
            const uint64_t same = __ballot(hold0 && vsel == val);
            rem &= ~same;
            if ((uint32_t)__popcll(same) > bestc) {
              bestc = (uint32_t)__popcll(same);
              hs = val;
            }
          }
          have_hs = true;
        }
      }
#pragma unroll
      for (int u = 0; u < kClassChunk; ++u) {
        const bool ex = hold[u] && v[u] != hs;
        const uint64_t em = __ballot(ex);
        const uint32_t k = nexc + (uint32_t)__popcll(em & ((1ull << lane) - 1ull));
        if (ex && k < kGroupHold) rec[1 + k] = make_uint2((uint32_t)((wb + w0 + u) * 64 + lane), v[u]);
        nexc += (uint32_t)__popcll(em);
      }
    }
  }
  return (nexc <= kGroupHold && hs > 0u && hs < (1u << 24)) ? ((nexc << 24) | hs) : kGroupNone;
}

// a wave-uniform 64-bit value in scalar registers
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Prefix groups, pass 2 (a persistent grid over the leaders' lists, which
// the claim pass wrote): the walk of the group's longest segment on every
// holder of its first block, into the slot's record (up to kGroupHold
// holders, each walked on its row) or a row of the popular area (more
// holders, walked together through the prefix index).
__global__ __launch_bounds__(64) void group_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  const int32_t nw = (a.n_inst + 63) >> 6;
  uint64_t* bmA = stage + kStage;
  uint64_t* bmN = bmA + nw;
  for (int32_t w = threadIdx.x; w < 2 * nw; w += 64) bmA[w] = 0ull;
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  const GroupTab& G = a.grp;
  // workgroup b takes entry (b / 64) * 8 + b % 8 of list (b / 8) % 8, then
  // every (grid / 8)-th after it: each list is spread over all XCDs (b runs
  // on XCD b % 8), so an XCD does not inherit one list's share of long walks
  static_assert(kXcds == 8, "the list walk maps workgroups to 8 lists");
  // (with Q waves per group, entry v of the list is part v % Q of group
  // v / Q)
  const uint32_t x = (blockIdx.x >> 3) & 7u;
  uint32_t groups = 0u, pmax = 0u;  // every list's length and longest segment (the same in every wave)
  for (int l = 0; l < kXcds; ++l) {
    const uint2 lw = *reinterpret_cast<const uint2*>(G.lctr + l * kListCtrWords);
    groups += lw.x;
    pmax = lw.y > pmax ? lw.y : pmax;
  }
  groups = (uint32_t)__builtin_amdgcn_readfirstlane((int)groups);
  pmax = (uint32_t)__builtin_amdgcn_readfirstlane((int)pmax);
  // no more parts than the longest segment fills (kGroupPartMin positions each)
  const uint32_t qp = (pmax + kGroupPartMin - 1u) / kGroupPartMin;
  uint32_t q0 = groups ? G.walkers / groups : 1u;
  q0 = q0 < qp ? q0 : qp;
  const uint32_t Q = q0 < 1u ? 1u : (q0 > kGroupSplitMax ? kGroupSplitMax : q0);
  const uint32_t nx = (uint32_t)__builtin_amdgcn_readfirstlane((int)G.lctr[x * kListCtrWords]) * Q;
  auto group_one = [&](uint32_t v, unsigned long long ent, unsigned long long plw, uint64_t key0) {
    const uint32_t part = v % Q;
    const uint32_t slot = (uint32_t)(ent & 0xFFFFFFull);
    const int64_t pre_off = (int64_t)(ent >> 24) - 1;
    const int32_t plen = (int32_t)(plw & ((1ull << kGroupGenShift) - 1ull));  // every member lies in the pool
    // this wave's part of the segment: [s0, s1), at least kGroupPartMin
    // positions and whole 512-position compare steps (a part costs its own
    // preamble of dependent reads)
    const int32_t step0 = (((plen + (int32_t)Q - 1) / (int32_t)Q) + 511) / 512 * 512;
    const int32_t step = step0 > kGroupPartMin ? step0 : kGroupPartMin;
    const int32_t s0 = (int32_t)part * step;
    const int32_t s1 = s0 + step < plen ? s0 + step : plen;
    if (part != 0u && s0 >= plen) return;  // (uniform: no workgroup barrier skipped)
    const ChainRef c{a.pool + pre_off, a.pool + pre_off, plen, plen};
    // (key0: the segment's first block, read beside its length; the
    // holders' row walks read the chain directly, only the index walk
    // stages its head)
    const IdxHit h0 = index_lookup(a.x, key0, g == 0, g, s);
    const bool found0 = __shfl(h0.found ? 1 : 0, 0) != 0;
    const uint32_t off0 = __shfl(h0.off, 0), cnt0 = __shfl(h0.cnt, 0);
    uint2* rec = G.rec + (size_t)slot * kGroupRec;
    uint32_t cnt = 0u;
    if (found0 && cnt0 > kGroupHold) {
      if (part != 0u) return;  // a popular group: one wave walks all holders
      if (cnt0 > kPopular && G.pop_pass &&
          (uint32_t)__builtin_amdgcn_readfirstlane((int)rec[kGroupClsWord].y) != kGroupUnlisted)
        return;  // listed by the claim pass: the popular pass's (it writes the record)
      const int32_t nst = plen < kStage ? plen : kStage;
      __syncthreads();  // (the previous index walk is done with the stage)
      for (int32_t j = lane; j < nst; j += 64) stage[j] = c.pre[j];
      __syncthreads();
      uint32_t row = 0;
      if (lane == 0) row = atomicAdd(G.pop_ctr, 1u);
      row = (uint32_t)__shfl((int)row, 0);
      cnt = kGroupNone;
      if (row < G.pop_cap) {
        // the live set: every holder of the first block
        if (cnt0 > kPopular) {
          const uint64_t* bm = a.x.bitmaps + (size_t)off0 * a.x.nw;
          for (int32_t w = lane; w < nw; w += 64) bmA[w] = bm[w];
        } else {
          for (uint32_t t = lane; t < cnt0; t += 64) {
            const uint32_t id = a.x.holders[off0 + t];
            atomicOr(reinterpret_cast<unsigned long long*>(&bmA[id >> 6]), 1ull << (id & 63));
          }
        }
        __syncthreads();
        uint32_t* hp = G.pop + (size_t)row * (size_t)a.n_inst;
        index_walk<true, true>(a, c, stage, bmA, bmN, nw, cnt0, 1,
                               [&](uint32_t id, uint32_t h) { hp[id] = h; }, lane, g, s);
        cnt = kGroupPop | row;
        const uint32_t clsw = cnt0 > kPopular ? popular_class(a, rec, hp, off0, nw, lane) : kGroupNone;
        if (lane == 0) rec[kGroupClsWord] = make_uint2(clsw, off0);
      }
    } else if (found0) {
      // the walk from s0 on the chain cut at s1: the first position there
      // whose block the holder lacks
      const ChainRef cp{c.pre, c.tail, s1, s1};
      const uint32_t id = (uint32_t)lane < cnt0 ? a.x.holders[off0 + lane] : 0u;
      uint32_t myhit = 0;
      for (uint32_t k = 0; k < cnt0; ++k) {
        const uint32_t idk = (uint32_t)__shfl((int)id, (int)k);
        // a group's segment is typically a long run: 512 positions per step
        const uint32_t hk =
            s0 < s1 ? run_walk<false, 8, 8>(a.t, idk, cp, nullptr, s0, g, s, s0 == 0 ? key0 : 0ull) : (uint32_t)s1;
        if ((uint32_t)lane == k) myhit = (int32_t)hk < s1 ? hk : (uint32_t)plen;  // no miss here: plen
      }
      if ((uint32_t)lane < cnt0) {
        if (Q == 1u) {
          rec[1 + lane] = make_uint2(id, myhit);
        } else {
          if (part == 0u) rec[1 + lane].x = id;
          atomicMin(&rec[1 + lane].y, myhit);
        }
      }
      cnt = cnt0;
    }
    if (lane == 0 && part == 0u) rec[0] = make_uint2((uint32_t)plen, cnt);
  };
  const uint32_t vstep = gridDim.x >> 3;
  const uint32_t vfirst = (blockIdx.x >> 6) * 8u + (blockIdx.x & 7u);
  // A group's first reads (its list entry, then its length word and first
  // block) are issued a group ahead (the entry two ahead): they arrive
  // while the group before walks.  Entries past the list's end read its
  // last entry instead (never used).
  auto entry_at = [&](uint32_t vv) -> unsigned long long {
    return G.lists[(size_t)x * G.lcap + (vv < nx ? vv : nx - 1u) / Q];
  };
  unsigned long long ent_c = 0ull, ent_n = 0ull, plw_c = 0ull;
  uint64_t key_c = 0ull;
  if (vfirst < nx) {
    ent_c = (unsigned long long)uniform64((int64_t)entry_at(vfirst));
    ent_n = entry_at(vfirst + vstep);
    plw_c = (unsigned long long)uniform64((int64_t)G.plen[(uint32_t)(ent_c & 0xFFFFFFull)]);
    key_c = (uint64_t)uniform64((int64_t)a.pool[(int64_t)(ent_c >> 24) - 1]);
  }
  for (uint32_t v = vfirst; v < nx; v += vstep) {
    // the next group's reads (ent_n arrived during this loop's last group)
    const unsigned long long ent_nu = (unsigned long long)uniform64((int64_t)ent_n);
    const unsigned long long plw_n = G.plen[(uint32_t)(ent_nu & 0xFFFFFFull)];
    const uint64_t key_n = a.pool[(int64_t)(ent_nu >> 24) - 1];
    const unsigned long long ent_nn = entry_at(v + 2u * vstep);
    group_one(v, ent_c, plw_c, key_c);
    ent_c = ent_nu;
    plw_c = (unsigned long long)uniform64((int64_t)plw_n);
    key_c = (uint64_t)uniform64((int64_t)key_n);
    ent_n = ent_nn;
  }
}

// ------------------------------------------------------------ popular pass
// Beside the walk pass (which runs on a second stream): the groups whose
// first block has a holder bitmap (more than kPopular holders; e.g. a
// 128-block system prompt held by nearly every instance).  The walk pass would walk each of
// them through the index, eight positions per pair of dependent reads, all
// over the same shared prefix.  Here the prefix is walked once per first
// block (by its representative, every position of a round at once), and
// each group starts from that walk at the end of its common prefix with the
// representative's segment.

// Word `lane` of the holder bitmap of an index entry's holder list (cnt <=
// kPopular ascending ids).
__device__ __forceinline__ uint64_t list_word(const GIndex& x, uint32_t off, uint32_t cnt, int lane) {
  const uint32_t idv = (uint32_t)lane < cnt ? (uint32_t)x.holders[off + (uint32_t)lane] : 0xFFFFFFFFu;
  uint64_t m = 0ull;
  for (uint32_t k = 0; k < cnt; ++k) {
    const uint32_t id = (uint32_t)__shfl((int)idv, (int)k);
    if ((id >> 6) == (uint32_t)lane) m |= 1ull << (id & 63u);
  }
  return m;
}

// Popular pass 1: one workgroup of kPrefixWaves waves per representative
// (the bitmaps whose representative word this window's claim pass set).
// Rounds of kPrefixWaves x 32 positions of its segment: wave w looks up its
// 32 positions (four lookups, then the 32 holder bitmaps, all in flight)
// and takes, for every holder of the first block, the first of them it
// lacks; the least over the waves (an LDS minimum) is the holder's first
// missing position, and the AND of the waves' survivors (LDS words) the
// holders with every position so far.  Rounds go on while more than one
// holder is left.  Row `pre` of the bitmap: that position, or ~0 for the
// holders that have all of them; pre_q: the round's end.  Pools of at most
// 64 x kPopWords instances (the live set is one bitmap word per lane).
constexpr int kPrefixWaves = 4;
constexpr int kPrefixSpan = 32;  // positions per wave and round
constexpr int32_t kPrefixMax = 1 << 14;

__global__ __launch_bounds__(64 * kPrefixWaves) void popular_prefix_kernel(ScoreArgs a) {
  __shared__ uint64_t stage[kStage];
  __shared__ uint32_t fmiss[64 * kPopWords];  // first missing position per instance (~0: none)
  __shared__ uint64_t firstw[kPopWords], livew[kPopWords];
  __shared__ uint2 reps[64 * kPrefixWaves];  // {bitmap, representative slot}
  __shared__ uint32_t n_reps, n_live;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = lane >> 3, s = lane & 7;
  const GroupTab& G = a.grp;
  const unsigned long long lmask = (1ull << kGroupGenShift) - 1ull;
  const int32_t nw = (a.n_inst + 63) >> 6;
  if (nw > kPopWords) return;
  const uint32_t tag = (uint32_t)(kGroupGenMax - G.gen);
  const uint32_t chunk = 64u * kPrefixWaves;
  for (uint32_t base = blockIdx.x * chunk; base < G.rep_cap; base += gridDim.x * chunk) {
    // the bitmaps of this chunk that first blocks of listed groups have
    if (tid == 0) n_reps = 0u;
    __syncthreads();
    const uint32_t bn = base + (uint32_t)tid;
    if (bn < G.rep_cap) {
      const unsigned long long rw = G.rep[bn];
      if ((uint32_t)(rw >> 32) == tag) reps[atomicAdd(&n_reps, 1u)] = make_uint2(bn, (uint32_t)rw);
    }
    __syncthreads();
    const uint32_t nr = n_reps;
    for (uint32_t r = 0; r < nr; ++r) {
      const uint2 ent = reps[r];
      const uint32_t off0 = ent.x, slot = ent.y;
      const int64_t pre_off = (int64_t)(G.keys[slot] & lmask) - 1;
      const int32_t plen = (int32_t)(G.plen[slot] & lmask);
      const int32_t lim = plen < kPrefixMax ? plen : kPrefixMax;
      const ChainRef c{a.pool + pre_off, a.pool + pre_off, plen, plen};
      const int32_t nst = plen < kStage ? plen : kStage;
      for (int32_t j = tid; j < nst; j += 64 * kPrefixWaves) stage[j] = c.pre[j];
      for (int32_t i = tid; i < 64 * nw; i += 64 * kPrefixWaves) fmiss[i] = 0xFFFFFFFFu;
      const uint64_t first = lane < nw ? a.x.bitmaps[(size_t)off0 * a.x.nw + lane] : 0ull;
      if (wv == 0 && lane < nw) {
        firstw[lane] = first;
        livew[lane] = first;
      }
      __syncthreads();
      int32_t p = 1;
      uint32_t nalive = 2u;
      while (p < lim && nalive > 1u) {
        const int32_t p0 = p + wv * kPrefixSpan;  // this wave's positions [p0, p0 + 32)
        constexpr int U = kPrefixSpan / 8;
        IdxHit hq[U];
        uint64_t kq[U];
        IdxEntry e[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int32_t jq = p0 + 8 * u + g;
          kq[u] = jq < lim ? (jq < kStage ? stage[jq] : chain_global(c, jq)) : 0ull;
          e[u] = kq[u] ? a.x.ent[(size_t)bucket_of(kq[u], kIndexSalt, a.x.shift) * kSlotsPerBucket + s]
                       : IdxEntry{0ull, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const uint64_t fm = __ballot(kq[u] != 0ull && e[u].key == kq[u]);
          const uint64_t em = __ballot(kq[u] != 0ull && e[u].key == 0ull);
          const uint32_t f = (uint32_t)(fm >> (8 * g)) & 0xFFu;
          const uint32_t z = (uint32_t)(em >> (8 * g)) & 0xFFu;
          const int src = 8 * g + (f ? __builtin_ctz(f) : 0);
          hq[u].found = f != 0u;
          hq[u].off = __shfl(e[u].off, src);
          hq[u].cnt = __shfl(e[u].cnt, src);
          if (__ballot(kq[u] != 0ull && !f && !z)) hq[u] = index_lookup(a.x, kq[u], kq[u] != 0ull, g, s);
        }
        uint64_t pw[kPrefixSpan];
#pragma unroll
        for (int t = 0; t < kPrefixSpan; ++t) {
          const bool f = __shfl(hq[t / 8].found ? 1 : 0, 8 * (t % 8)) != 0;
          const uint32_t off = __shfl(hq[t / 8].off, 8 * (t % 8)), cnt = __shfl(hq[t / 8].cnt, 8 * (t % 8));
          pw[t] = f && cnt > kPopular && lane < nw ? a.x.bitmaps[(size_t)off * a.x.nw + lane] : 0ull;
        }
        // the first of this wave's positions each holder lacks
        uint64_t have = first;
#pragma unroll
        for (int t = 0; t < kPrefixSpan; ++t) {
          if (p0 + t < lim) {
            const bool f = __shfl(hq[t / 8].found ? 1 : 0, 8 * (t % 8)) != 0;
            const uint32_t off = __shfl(hq[t / 8].off, 8 * (t % 8)), cnt = __shfl(hq[t / 8].cnt, 8 * (t % 8));
            const uint64_t keep = !f ? 0ull : (cnt > kPopular ? pw[t] : list_word(a.x, off, cnt, lane));
            uint64_t d = have & ~keep;
            if (__ballot(__popcll(d) > 4u)) {  // many leave here: lanes over each word's bits
              for (int32_t w = 0; w < nw; ++w) {
                const uint64_t dw = (uint64_t)lane_value64((int64_t)d, w);
                if ((dw >> lane) & 1ull) atomicMin(&fmiss[w * 64 + lane], (uint32_t)(p0 + t));
              }
            } else {
              while (d) {
                const int b = __builtin_ctzll(d);
                d &= d - 1ull;
                atomicMin(&fmiss[lane * 64 + b], (uint32_t)(p0 + t));
              }
            }
            have &= keep;
          }
        }
        if (lane < nw) atomicAnd(reinterpret_cast<unsigned long long*>(&livew[lane]), have);
        __syncthreads();
        if (wv == 0) {  // holders with every position so far
          const uint32_t cnt = wave_sum_u32(lane < nw ? (uint32_t)__popcll(livew[lane]) : 0u);
          if (lane == 0) n_live = cnt;
        }
        __syncthreads();
        nalive = n_live;
        p = p + kPrefixWaves * kPrefixSpan < lim ? p + kPrefixWaves * kPrefixSpan : lim;
      }
      // row of the bitmap: the holders' first missing positions
      uint32_t* row = G.pre + (size_t)off0 * (size_t)a.n_inst;
      for (int32_t i = tid; i < a.n_inst; i += 64 * kPrefixWaves)
        if ((firstw[i >> 6] >> (i & 63)) & 1ull) row[i] = fmiss[i];
      if (tid == 0) G.pre_q[off0] = (uint32_t)p;
      __syncthreads();
    }
  }
}

// Popular pass 2 (a persistent grid over plist): listed group v.  Its
// segment and its representative's agree on their first k blocks
// (compared here; k at most the prefix walk's end), so a holder whose first
// missing position there is h < k has hit h here too, and the others hold
// the first k blocks: only they are walked on, from k, through the index
// (one holder left: along its row, 512 positions per step).  Then the
// record, as the walk pass writes it, with popular row pop_cap + v.
constexpr int kMemberChunk = 16;  // bitmap words whose holders' hits are read together
constexpr int kPopPrefixGrid = 64;   // workgroups of its prefix kernel
constexpr int kPopWalkGrid = 4096;   // waves of its member kernel

__global__ __launch_bounds__(64) void popular_member_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  const int32_t nw = (a.n_inst + 63) >> 6;
  uint64_t* bmA = stage + kStage;
  uint64_t* bmN = bmA + nw;
  for (int32_t w = threadIdx.x; w < 2 * nw; w += 64) bmA[w] = 0ull;
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  const GroupTab& G = a.grp;
  const unsigned long long lmask = (1ull << kGroupGenShift) - 1ull;
  if (nw > kPopWords) return;
  uint32_t n = (uint32_t)__builtin_amdgcn_readfirstlane((int)G.lctr[kPopCountWord]);
  n = n < G.plist_cap ? n : G.plist_cap;
  for (uint32_t v = blockIdx.x; v < n; v += gridDim.x) {
    const uint2 ent = G.plist[v];
    const uint32_t slot = ent.x, off0 = ent.y;
    const int64_t pre_off = (int64_t)(G.keys[slot] & lmask) - 1;
    const int32_t plen = (int32_t)(G.plen[slot] & lmask);
    const uint32_t rslot = (uint32_t)G.rep[off0];  // this window's: every listed group set its tag
    const uint32_t q = G.pre_q[off0];
    const uint64_t myw = lane < nw ? a.x.bitmaps[(size_t)off0 * a.x.nw + lane] : 0ull;  // word `lane`
    const ChainRef c{a.pool + pre_off, a.pool + pre_off, plen, plen};
    const int32_t nst = plen < kStage ? plen : kStage;
    __syncthreads();
    for (int32_t j = lane; j < nst; j += 64) stage[j] = c.pre[j];
    const int64_t rpre = (int64_t)(G.keys[rslot] & lmask) - 1;
    const int32_t rlen = (int32_t)(G.plen[rslot] & lmask);
    uint2* rec = G.rec + (size_t)slot * kGroupRec;
    const uint32_t row = G.pop_cap + v;
    uint32_t* hp = G.pop + (size_t)row * (size_t)a.n_inst;
    // k: the common prefix of the two segments, at most the prefix walk's end
    int32_t lim = plen < rlen ? plen : rlen;
    lim = lim < (int32_t)q ? lim : (int32_t)q;
    int32_t k = lim;
    if (rslot != slot) {
      const uint64_t* rc = a.pool + rpre;
      for (int32_t j0 = 0; j0 < lim; j0 += 64 * 8) {
        uint32_t firstm = ~0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int32_t j = j0 + u * 64 + lane;
          if (j < lim && c.pre[j] != rc[j] && (uint32_t)j < firstm) firstm = (uint32_t)j;
        }
        firstm = wave_min_u32(firstm);
        if (firstm != ~0u) {
          k = (int32_t)firstm;
          break;
        }
      }
    }
    // the live set at k; the holders missing a position before k keep it
    const uint32_t* prow = G.pre + (size_t)off0 * (size_t)a.n_inst;
    uint32_t nalive = 0u;
    for (int32_t w0 = 0; w0 < nw; w0 += kMemberChunk) {
      uint32_t h[kMemberChunk];
#pragma unroll
      for (int u = 0; u < kMemberChunk; ++u) {
        const uint64_t word = (uint64_t)lane_value64((int64_t)myw, (w0 + u) & 63);
        const bool hold = w0 + u < nw && ((word >> lane) & 1ull) != 0ull;
        h[u] = hold ? prow[(w0 + u) * 64 + lane] : 0u;
      }
#pragma unroll
      for (int u = 0; u < kMemberChunk; ++u) {
        const uint64_t word = (uint64_t)lane_value64((int64_t)myw, (w0 + u) & 63);
        const bool hold = w0 + u < nw && ((word >> lane) & 1ull) != 0ull;
        const bool live = hold && h[u] >= (uint32_t)k;
        if (hold && !live) hp[(w0 + u) * 64 + lane] = h[u];
        const uint64_t lw = __ballot(live);
        if (lane == 0 && w0 + u < nw) bmA[w0 + u] = lw;
        nalive += (uint32_t)__popcll(lw);
      }
    }
    __syncthreads();
    index_walk<true, true, 8, 4, true>(a, c, stage, bmA, bmN, nw, nalive, k,
                                 [&](uint32_t id, uint32_t hh) { hp[id] = hh; }, lane, g, s);
    const uint32_t clsw = popular_class(a, rec, hp, off0, nw, lane);
    if (lane == 0) {
      rec[kGroupClsWord] = make_uint2(clsw, off0);
      rec[0] = make_uint2((uint32_t)plen, kGroupPop | row);
    }
  }
}

// LDS of one scoring wave: chain stage | live bitmap | next bitmap |
// candidate bitmap (instances holding the first block) | group hits and ids
// of up to 64 candidates | u16 hit slots (or device scratch for large
// pools) | for pools of at most 64 instances (SMALL) the rooms, states and
// zero-hit thresholds, copied once per launch.
constexpr int32_t kSmallPool = 64;

constexpr int32_t kBatch = 4;  // most requests whose inputs one wave loads together
// Bytes of the batch buffers: group records, descriptors, group slots,
// deferral marks (a multiple of 16).
// the general kernel's batch buffers: with the hand-over lists a wave loads
// up to kListBatch entries of its share together
constexpr int32_t kListBatch = 16;
constexpr size_t kBatchLds = (size_t)kListBatch * (kGroupRec * 8 + 3 * 8 + 4 + 4);
// Result flag of a request the lean scoring kernel left to the general one
// (never returned: the general kernel overwrites the result).
constexpr uint32_t kDeferred = 0x80000000u;
static_assert(kBatchLds % 16 == 0, "batch buffers keep the LDS layout 16-byte aligned");

__host__ __device__ inline size_t score_lds_base(int32_t n_inst, bool hits_in_lds) {
  const size_t nw = ((size_t)n_inst + 63) / 64;
  const size_t hits = hits_in_lds ? (size_t)n_inst * sizeof(uint16_t) : 0;
  const size_t b = (size_t)kStage * sizeof(uint64_t) + 3 * nw * sizeof(uint64_t) +
                   64 * sizeof(uint32_t) + 64 * sizeof(uint16_t) + hits;
  return (b + 15) / 16 * 16;
}

// The general scorer: every request (groups or not, every selector), or
// with a.defer_only only the requests the lean scorer marked kDeferred.
// FAST: the policy the four-requests-per-wave scorer serves (keyed
// selector, monotone model, no TTFT admission, no set sizes), so the
// other policies' paths compile away.
template <bool HITS_IN_LDS, bool SMALL, bool FAST>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void score_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int32_t n_inst = a.n_inst;
  const int32_t nw = (n_inst + 63) >> 6;
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  uint64_t* bmA = stage + kStage;
  uint64_t* bmN = bmA + nw;
  uint64_t* bmC = bmN + nw;
  uint32_t* ch = reinterpret_cast<uint32_t*>(bmC + nw);  // group hits of the candidates
  uint16_t* cl = reinterpret_cast<uint16_t*>(ch + 64);
  uint16_t* hits = HITS_IN_LDS ? cl + 64 : a.scratch + (size_t)blockIdx.x * (size_t)n_inst;
  uint2* lrec = reinterpret_cast<uint2*>(smem + score_lds_base(n_inst, HITS_IN_LDS));
  int64_t* lq64 = reinterpret_cast<int64_t*>(lrec + kListBatch * kGroupRec);
  uint32_t* lgso = reinterpret_cast<uint32_t*>(lq64 + 3 * kListBatch);
  uint32_t* ldef = lgso + kListBatch;
  int64_t* lroom = reinterpret_cast<int64_t*>(ldef + kListBatch);
  InstState* linst = reinterpret_cast<InstState*>(lroom + kSmallPool);
  int4* llm = reinterpret_cast<int4*>(linst + kSmallPool);
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  // With the hand-over lists, only the listed requests: lane l holds the
  // running total of the sub-lists' lengths through sub-list l.  (Reading
  // the model and window constants before the test costs the empty pass
  // more than it saves a full one.)
  const bool listed = a.defer_only && a.dlist != nullptr;
  uint32_t lincl = listed ? a.dcnt[lane * kDeferStride] : 0u;
  const uint32_t dany = !listed && a.defer_only ? *a.defer_any : 1u;

  static_assert(kDeferLists == 64, "one sub-list per lane");
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = (uint32_t)__shfl_up((int)lincl, d);
    if (lane >= d) lincl += o;
  }
  const uint32_t n_listed = (uint32_t)__builtin_amdgcn_readlane((int)lincl, 63);
  if (listed ? n_listed == 0u : dany == 0u) return;  // nothing was left
  __shared__ DevModel lmodel;
  stage_model(lmodel, a.model, lane, 64);
  // FAST (pools of at most 4,096 instances: at most 64 chunks of the key
  // order): the chunk summaries and threshold maxima, window constants, in
  // LDS for the whole launch
  __shared__ uint4 lcsum[FAST ? 64 : 1];
  __shared__ int32_t llm1v[FAST ? 64 : 1];
  if (FAST) {
    const int32_t n1c = (n_inst + 63) >> 6;
    lcsum[lane] = lane < n1c ? a.csum[lane] : make_uint4(0u, 0u, 0u, 0u);
    llm1v[lane] = lane < n1c ? a.lm1[lane] : -1;
  }
  // entry i of the concatenated sub-lists (per lane; every lane takes part)
  auto listed_req = [&](uint32_t i) -> int32_t {
    int q = 0;  // sub-lists that end at or before i
#pragma unroll
    for (int step = 32; step >= 1; step >>= 1)
      if ((uint32_t)__shfl((int)lincl, q + step - 1) <= i) q += step;
    const uint32_t before = (uint32_t)__shfl((int)lincl, q > 0 ? q - 1 : 0);
    return a.dlist[(size_t)q * (size_t)a.dcap + (i - (q > 0 ? before : 0u))];
  };
  __syncthreads();
  const DevModel& m = lmodel;
  uint32_t* const sizes = FAST ? nullptr : a.sizes;
  const bool sel_hcq = !FAST && m.sel == PS_SEL_HCQ;
  const bool sel_random = !FAST && m.sel == PS_SEL_RANDOM;
  auto room_of = [&](uint32_t i) -> int64_t { return SMALL ? lroom[i] : a.room[i]; };
  auto state_of = [&](uint32_t i) -> InstState { return SMALL ? linst[i] : a.inst[i]; };

  for (int32_t w = lane; w < 3 * nw; w += 64) bmA[w] = 0ull;
  if (SMALL) {
    if (lane < n_inst) {
      lroom[lane] = a.room[lane];
      linst[lane] = a.inst[lane];
      llm[lane] = a.lm[lane];
    }
    __syncthreads();
  }

  // Requests are taken in batches of a.batch (<= kBatch) consecutive ones: their
  // descriptors and group slots arrive with one round trip, their group
  // records with a second, into LDS; then each is scored from there.
  // Listed: this wave takes every gridDim.x-th entry of the concatenated
  // sub-lists from entry blockIdx.x (equal shares; entries of one group,
  // which cost alike, spread over the waves), in batches of kBatch (its
  // entries read 64 at a time into lanes); otherwise batches of
  // consecutive requests, every gridDim.x-th batch.
  const int32_t B = listed ? kListBatch : a.batch;
  const int32_t k_lo = listed ? 0 : blockIdx.x * B;
  const int32_t k_hi = !listed ? a.n_req
                       : n_listed > blockIdx.x ? (int32_t)((n_listed - 1u - blockIdx.x) / gridDim.x) + 1 : 0;
  const int32_t k_step = listed ? B : (int32_t)gridDim.x * B;
  int32_t lbase = k_lo - 64, litem = 0;  // listed: this wave's entries lbase .. lbase + 63 in litem
  for (int32_t rb = k_lo; rb < k_hi; rb += k_step) {
    const int32_t nb = k_hi - rb < B ? k_hi - rb : B;
    int32_t rq = rb + lane;  // the request of the batch's entry `lane` (lane < nb)
    if (listed) {
      if (rb + nb > lbase + 64) {
        lbase = rb;
        const uint32_t i = blockIdx.x + gridDim.x * (uint32_t)(lbase + lane);
        const int32_t v = listed_req(i < n_listed ? i : n_listed - 1u);
        litem = lbase + lane < k_hi ? v : 0;
      }
      rq = __shfl(litem, (rb - lbase + lane) & 63);
    }
    const int32_t rq3 = __shfl(rq, lane < 3 * nb ? lane / 3 : 0);
    __syncthreads();  // the previous batch is done with the batch buffers
    if (lane < nb) {
      lgso[lane] = a.grp.keys ? a.grp.slot_of[rq] : kGroupNoSlot;
      if (a.defer_only) ldef[lane] = listed ? kDeferred : a.out[rq].flags & kDeferred;
    }
    if (lane < 3 * nb) lq64[lane] = reinterpret_cast<const int64_t*>(a.reqs + rq3)[lane % 3];
    __syncthreads();
    // the records' words, three loads in flight per lane (loads at slot 0
    // stand in for requests without one)
    for (int32_t w0 = lane; w0 < nb * kGroupRec; w0 += 3 * 64) {
      uint2 rv[3];
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int32_t w = w0 + 64 * u;
        const uint32_t so = w < nb * kGroupRec ? lgso[w / kGroupRec] : kGroupNoSlot;
        rv[u] = a.grp.rec[(size_t)(so != kGroupNoSlot ? so & ~kGroupLead : 0u) * kGroupRec + (uint32_t)(w % kGroupRec)];
      }
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int32_t w = w0 + 64 * u;
        if (w < nb * kGroupRec && lgso[w / kGroupRec] != kGroupNoSlot) lrec[w] = rv[u];
      }
    }
    __syncthreads();
    for (int32_t b = 0; b < nb; ++b) {
      const int32_t r = __builtin_amdgcn_readlane(rq, b);
      if (a.defer_only && __builtin_amdgcn_readfirstlane((int)ldef[b]) == 0) continue;
      // wave-uniform values read from LDS are moved to scalar registers
      const uint32_t gso = (uint32_t)__builtin_amdgcn_readfirstlane((int)lgso[b]);
      const ps_req ql = reinterpret_cast<const ps_req*>(lq64)[b];
      const ps_req q{uniform64(ql.pre_off), uniform64(ql.tail_off),
                     __builtin_amdgcn_readfirstlane(ql.pre_len),
                     __builtin_amdgcn_readfirstlane(ql.tail_len)};
      if (!req_valid(q, a.pool_len)) {
        if (lane == 0) {
          a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_INVALID};
          if (sizes) sizes[3 * (size_t)r] = sizes[3 * (size_t)r + 1] = sizes[3 * (size_t)r + 2] = 0;
        }
        continue;
      }
      const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
      const int32_t ell = c.len;
      const int64_t L = (int64_t)ell * m.bs;
      const float Lf = (float)L;
      // The group record (meta and up to 16 holders); a request with a
      // group result needs no staged chain.
      GroupMeta gm{0, kGroupNone};
      uint2 hd = make_uint2(0u, 0u);
      if (gso != kGroupNoSlot) {
        const uint2* grec = lrec + b * kGroupRec;
        const uint2 m0 = grec[0];
        if ((uint32_t)lane < kGroupHold) hd = grec[1 + lane];
        gm = GroupMeta{__builtin_amdgcn_readfirstlane((int)m0.x),
                       (uint32_t)__builtin_amdgcn_readfirstlane((int)m0.y)};
      }
      const bool grp = gm.cnt != kGroupNone;
      const bool gpop = grp && (gm.cnt & kGroupPop) != 0u;  // holders from the index
      // A popular group whose holders share one hit H* (but for at most
      // kGroupHold exceptions): the exceptions are candidates of their own,
      // the other holders one class (hit H*, one penalty, the first member of
      // T in key order found by a scan of the key-ordered states), the
      // non-holders the zero-hit class.  When no candidate is in T, the
      // fallback key is the minimum over C: the exceptions in it and the
      // eligible members of the admitted classes, scanned in id order.  When
      // a class's eligibility cannot be told from the 64 largest rooms, the
      // request takes the general path below.
      if (FAST && gpop) {
        const uint2 cwd = lrec[b * kGroupRec + kGroupClsWord];
        const uint32_t clsw = (uint32_t)__builtin_amdgcn_readfirstlane((int)cwd.x);
        const uint32_t hs = clsw & 0xFFFFFFu, nexc = clsw >> 24;
        const int32_t p0 = q.pre_len < gm.plen ? q.pre_len : gm.plen;
        if (clsw != kGroupNone && (int32_t)hs < p0) {
          // the holder bitmap, copied to LDS (bmA: free outside the index
          // walk, which sets it first): the class scan tests one bit per
          // instance
          const uint64_t* hg = a.x.bitmaps + (size_t)__builtin_amdgcn_readfirstlane((int)cwd.y) * a.x.nw;
          for (int32_t w = lane; w < nw; w += 64) bmA[w] = hg[w];
          const uint64_t* hb = bmA;
          const TopRoom trm = a.rtop[lane];
          // exceptions: state, eligibility, hit (resumed where it reaches p0)
          const bool eact = (uint32_t)lane < nexc;
          const uint32_t eid = eact ? hd.x : 0u;
          uint32_t ehit = eact ? hd.y : 0u;
          InstState est{};
          if (eact) {
            est = state_of(eid);
            atomicOr(reinterpret_cast<unsigned long long*>(&bmC[eid >> 6]), 1ull << (eid & 63));
          }
          const bool eel = eact && eligible(m, est.A1, est.S, L);
          __syncthreads();
          uint64_t need = __ballot(eel && (int32_t)ehit >= p0);
          while (need) {
            const int k = __builtin_ctzll(need);
            need &= need - 1;
            const uint32_t hk = run_walk<false>(a.t, (uint32_t)__shfl((int)eid, k), c, nullptr, p0, g, s);
            if (lane == k) ehit = hk;
          }
          const int64_t room0 = lane_value64(trm.room, 0), room63 = lane_value64(trm.room, 63);
          const bool topel = trm.room >= L;
          const bool thold = test_bit(hb, (uint32_t)trm.id);
          const bool texc = test_bit(bmC, (uint32_t)trm.id);
          const bool anyK = __ballot(topel && thold && !texc) != 0ull;
          const bool any0 = __ballot(topel && !thold) != 0ull;
          // with the 64th room eligible, a class absent from the top rooms may
          // still have eligible members
          bool decided = false;
          ps_result res{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
          if (!(room0 >= L)) {
            decided = true;  // A is empty
          } else if (!(room63 >= L) || (anyK && any0)) {
            const float Z = recompute_raw(m, Lf, Lf);
            const float W0 = fmaxf(0.0f, Z);
            const int64_t cK = (int64_t)hs * m.bs;
            const float WK = fmaxf(0.0f, recompute_raw(m, (float)(L - cK), Lf));
            uint32_t wb = 0x7F800000u;
            if (eel) wb = __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)ehit * m.bs), Lf)));
            if (lane == 0 && any0) wb = wb < __float_as_uint(W0) ? wb : __float_as_uint(W0);
            if (lane == 1 && anyK) wb = wb < __float_as_uint(WK) ? wb : __float_as_uint(WK);
            const float wmin = __uint_as_float(wave_min_u32(wb));
            const float slo = fmaxf(m.ttft_floor, t_prefill(m, Lf, 0.0f));
            const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
            const bool admitK = anyK && (!kvc || (WK - wmin) / Z <= m.eta);
            const bool admit0 = any0 && (!kvc || (W0 - wmin) / Z <= m.eta);
            Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
            if (eel) evaluate_with<true>(m, acc, eid, ehit, [&]() { return est; }, L, Lf, wmin, Z, kvc, slo);
            if (admitK) {  // the class's first member of T in key order
              const float nK = (float)(L - cK), cKf = (float)cK;
              // chunks of 64 key-ordered instances that may hold one: some
              // room holds L, and (monotone model: TPOT is at least t_iter
              // at L = 0, plus the class's interference when A1 > 1) some
              // lower bound passes the TPOT test; two chunks in flight
              const bool notpot = (m.flags & PS_F_NO_TPOT_FILTER) != 0u;
              const float xK = t_prefill(m, nK, cKf) / m.lout1;
              const int32_t n1 = (n_inst + 63) >> 6;
              bool found = false;
              for (int32_t c0 = 0; c0 < n1 && !found; c0 += 64) {
                const int32_t cc = c0 + lane;
                bool may = false;
                if (cc < n1) {
                  const uint4 cs = FAST ? lcsum[cc] : a.csum[cc];
                  const int64_t rmx = (int64_t)(((uint64_t)cs.w << 32) | cs.z);
                  may = rmx >= L && (notpot || __uint_as_float(cs.x) + xK < m.tau ||
                                     __uint_as_float(cs.y) < m.tau);
                }
                uint64_t cm = __ballot(may);
                while (cm && !found) {
                  int32_t kc[2];
                  kc[0] = c0 + __builtin_ctzll(cm);
                  cm &= cm - 1;
                  kc[1] = cm ? c0 + __builtin_ctzll(cm) : -1;
                  if (cm) cm &= cm - 1;
                  uint32_t i[2];
                  InstState st[2];
#pragma unroll
                  for (int u = 0; u < 2; ++u) {
                    const int32_t k = kc[u] * 64 + lane;
                    i[u] = 0u;
                    st[u] = InstState{};
                    if (kc[u] >= 0 && k < n_inst) {
                      i[u] = a.order0[k];
                      st[u] = a.inst_key[k];
                    }
                  }
#pragma unroll
                  for (int u = 0; u < 2; ++u) {
                    const int32_t k = kc[u] * 64 + lane;
                    const bool ok = kc[u] >= 0 && k < n_inst && test_bit(hb, i[u]) && !test_bit(bmC, i[u]) &&
                                    eligible(m, st[u].A1, st[u].S, L) &&
                                    (notpot || latency(m, st[u], nK, cKf, L).tpot < m.tau);
                    const uint64_t om = __ballot(ok);
                    if (!found && om) {
                      if (lane == __builtin_ctzll(om)) {
                        const uint64_t kt = select_key(m.sel, st[u], hs, i[u], 0ull);
                        acc.keyT = kt < acc.keyT ? kt : acc.keyT;
                      }
                      found = true;
                    }
                  }
                }
              }
            }
            if (admit0) {  // the zero-hit class's first member of T: thresholds
              const int32_t n1 = (n_inst + 63) >> 6;
              bool found = false;
              for (int32_t c0 = 0; c0 < n1 && !found; c0 += 64) {
                const int32_t cc = c0 + lane;
                uint64_t cm = __ballot(cc < n1 && (SMALL || (FAST ? llm1v[cc] : a.lm1[cc]) >= ell));
                while (cm && !found) {
                  const int32_t k = (c0 + __builtin_ctzll(cm)) * 64 + lane;
                  cm &= cm - 1;
                  const int4 e = k < n_inst ? (SMALL ? llm[k] : a.lm[k]) : make_int4(-1, 0, 0, 0);
                  const uint64_t om = __ballot(e.x >= ell && !test_bit(hb, (uint32_t)e.y));
                  if (om) {
                    if (lane == __builtin_ctzll(om)) {
                      InstState st{};
                      st.D = e.z;
                      st.Q = e.w;
                      const uint64_t kt = select_key(m.sel, st, 0u, (uint32_t)e.y, 0ull);
                      acc.keyT = kt < acc.keyT ? kt : acc.keyT;
                    }
                    found = true;
                  }
                }
              }
            }
            const uint64_t keyT = wave_min_u64(acc.keyT);
            uint64_t keyF = ~0ull;
            if (keyT == ~0ull) {
              // T is empty: the fallback key over C, whose members outside
              // the exceptions are the eligible members of the admitted
              // classes (the exceptions' keys are in acc.keyF); instances in
              // id order, two chunks of 64 states in flight
              const int64_t nKt = L - cK;
              for (int32_t base = 0; base < n_inst; base += 128) {
                InstState st[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                  const int32_t i = base + 64 * u + lane;
                  st[u] = i < n_inst ? state_of((uint32_t)i) : InstState{};
                }
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                  const uint32_t i = (uint32_t)(base + 64 * u + lane);
                  if ((int32_t)i < n_inst && !test_bit(bmC, i) && eligible(m, st[u].A1, st[u].S, L)) {
                    const bool hold = test_bit(hb, i);
                    if (hold ? admitK : admit0) {
                      const uint32_t v = hold ? hs : 0u;
                      const uint64_t lm = (uint64_t)(st[u].P + (hold ? nKt : L)) * (uint64_t)st[u].A1;
                      const uint64_t kf = (m.flags & PS_F_FALLBACK_DCQ) ? dcq_key(st[u], v, i) : ((lm << 16) | i);
                      acc.keyF = kf < acc.keyF ? kf : acc.keyF;
                    }
                  }
                }
              }
              keyF = wave_min_u64(acc.keyF);
            }
            if (keyT != ~0ull || keyF != ~0ull) {  // (neither: a non-finite model; the general path decides)
              const bool t = keyT != ~0ull;
              const uint32_t best = (uint32_t)((t ? keyT : keyF) & 0xFFFFu);
              const uint64_t em = __ballot(eact && eid == best);
              const uint32_t ev = (uint32_t)__shfl((int)ehit, em ? __builtin_ctzll(em) : 0);
              const uint32_t v = em ? ev : test_bit(hb, best) ? hs : 0u;
              const int64_t c_tok = (int64_t)v * m.bs;
              const Lat lt = latency(m, state_of(best), (float)(L - c_tok), (float)c_tok, L);
              res = ps_result{(int32_t)best, (int32_t)v, lt.ttft, lt.tpot,
                              (t ? 0u : PS_R_FALLBACK) | (lt.ttft > slo ? PS_R_TTFT_MISS : 0u)};
              decided = true;
            }
          }
          __syncthreads();
          if (eact) bmC[eid >> 6] = 0ull;
          __syncthreads();
          if (decided) {
            if (lane == 0) a.out[r] = res;
            continue;
          }
        }
      }
      const int32_t nst = grp ? 0 : (ell < kStage ? ell : kStage);
      // The chain head's loads and the room search's are in flight together.
      uint64_t sv[kStage / 64];
  #pragma unroll
      for (int u = 0; u < kStage / 64; ++u) {
        const int32_t j = lane + 64 * u;
        sv[u] = j < nst ? chain_global(c, j) : 0ull;
      }
      // |A|: capacity-eligible instances are those with room >= L.
      const uint32_t nA =
          SMALL ? (uint32_t)__popcll(__ballot(lane < n_inst && lroom[lane] >= L))
                : (uint32_t)(n_inst - wave_lower_bound(a.room_sorted, n_inst, L, lane));
      if (!grp) {
        __syncthreads();
  #pragma unroll
        for (int u = 0; u < kStage / 64; ++u) {
          const int32_t j = lane + 64 * u;
          if (j < nst) stage[j] = sv[u];
        }
        __syncthreads();
      }

      // (1) Holders of the first block among the eligible instances.
      uint32_t nCand = 0;
      if (grp && !gpop) {  // from the group record: ids and hits of the shared segment
        const bool el = nA > 0 && (uint32_t)lane < gm.cnt && room_of(hd.x) >= L;
        const uint64_t em = __ballot(el);
        const uint32_t rank = (uint32_t)__popcll(em & lt_mask);
        if (el) {
          cl[rank] = (uint16_t)hd.x;
          ch[rank] = hd.y;
          atomicOr(reinterpret_cast<unsigned long long*>(&bmC[hd.x >> 6]), 1ull << (hd.x & 63));
        }
        nCand = (uint32_t)__popcll(em);
      } else if (nA > 0 && ell > 0) {
        const IdxHit h0 = index_lookup(a.x, grp ? c.pre[0] : stage[0], g == 0, g, s);
        const bool found0 = __shfl(h0.found ? 1 : 0, 0) != 0;
        const uint32_t off0 = __shfl(h0.off, 0), cnt0 = __shfl(h0.cnt, 0);
        if (found0 && cnt0 > kPopular) {  // holders as a bitmap: lanes over the pool
          // 64 instances per step, rooms read coalesced, four steps in flight
          const uint64_t* bm = a.x.bitmaps + (size_t)off0 * a.x.nw;
          for (int32_t w0 = 0; w0 < nw; w0 += 4) {
            bool el[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int32_t w = w0 + u;
              const int32_t i = w * 64 + lane;
              el[u] = w < nw && i < n_inst && ((bm[w] >> lane) & 1ull) && room_of((uint32_t)i) >= L;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int32_t w = w0 + u;
              const uint64_t em = __ballot(el[u]);
              if (w < nw && lane == 0) bmC[w] = em;
              const uint32_t rank = nCand + (uint32_t)__popcll(em & lt_mask);
              if (el[u] && rank < 64) cl[rank] = (uint16_t)(w * 64 + lane);
              nCand += (uint32_t)__popcll(em);
            }
          }
        } else if (found0) {
          for (uint32_t t0 = 0; t0 < cnt0; t0 += 64) {
            const uint32_t t = t0 + lane;
            const uint32_t id = t < cnt0 ? a.x.holders[off0 + t] : 0u;
            const bool el = t < cnt0 && room_of(id) >= L;
            const uint64_t em = __ballot(el);
            const uint32_t rank = nCand + (uint32_t)__popcll(em & lt_mask);
            if (el) {
              if (rank < 64) cl[rank] = (uint16_t)id;
              atomicOr(reinterpret_cast<unsigned long long*>(&bmC[id >> 6]), 1ull << (id & 63));
            }
            nCand += (uint32_t)__popcll(em);
          }
        }
      }
      __syncthreads();
      const bool few = nCand <= 64;

      // Walks.  few: each holder on its own table; else: all live holders
      // through the index, one position at a time.
      uint32_t myid = 0, myhit = 0;
      if (few && grp) {
        // Hit H of the shared segment: exact below the request's segment
        // length p; otherwise the walk resumes on its own chain at p.
        const int32_t p0 = q.pre_len < gm.plen ? q.pre_len : gm.plen;
        if ((uint32_t)lane < nCand) {
          myid = cl[lane];
          myhit = gpop ? a.grp.pop[(size_t)(gm.cnt & ~kGroupPop) * (size_t)n_inst + myid] : ch[lane];
        }
        uint64_t need = __ballot((uint32_t)lane < nCand && (int32_t)myhit >= p0);
        while (need) {
          const int k = __builtin_ctzll(need);
          need &= need - 1;
          const uint32_t id = (uint32_t)__shfl((int)myid, k);
          const uint32_t hk = run_walk<false>(a.t, id, c, nullptr, p0, g, s);
          if (lane == k) myhit = hk;
        }
        if ((uint32_t)lane < nCand) hits[myid] = encode_hit(myhit);
      } else if (few) {
        if ((uint32_t)lane < nCand) myid = cl[lane];
        for (uint32_t k = 0; k < nCand; ++k) {
          const uint32_t id = (uint32_t)__shfl((int)myid, (int)k);
          const uint32_t hk = ell > 1 ? run_walk<true>(a.t, id, c, stage, 0, g, s) : 1u;
          if ((uint32_t)lane == k) myhit = hk;
        }
        if ((uint32_t)lane < nCand) hits[myid] = encode_hit(myhit);
      } else if (!grp) {
        for (int32_t w = lane; w < nw; w += 64) bmA[w] = bmC[w];
        __syncthreads();
        index_walk<true, false>(a, c, stage, bmA, bmN, nw, nCand, 1,
                                [&](uint32_t id, uint32_t h) { hits[id] = encode_hit(h); }, lane, g, s);
      } else {
        // many candidates with a popular group's result: lanes over the
        // pool, resumes walked one at a time
        const uint32_t* hp = a.grp.pop + (size_t)(gm.cnt & ~kGroupPop) * (size_t)n_inst;
        const int32_t p0 = q.pre_len < gm.plen ? q.pre_len : gm.plen;
        for (int32_t base = 0; base < n_inst; base += 256) {  // four steps in flight
          bool cand[4];
          uint32_t v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int32_t i = base + 64 * u + lane;
            cand[u] = i < n_inst && test_bit(bmC, (uint32_t)i);
            v[u] = cand[u] ? hp[i] : 0u;
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            uint64_t need = __ballot(cand[u] && (int32_t)v[u] >= p0);
            while (need) {
              const int k = __builtin_ctzll(need);
              need &= need - 1;
              const uint32_t hk = run_walk<false>(a.t, (uint32_t)(base + 64 * u + k), c, nullptr, p0, g, s);
              if (lane == k) v[u] = hk;
            }
            if (cand[u]) hits[base + 64 * u + lane] = encode_hit(v[u]);
          }
        }
        __syncthreads();
      }

      // (2)-(3) Minimum recomputation penalty over A.  Every eligible
      // non-holder has hit 0 and the penalty W(n = L).
      const float Z = recompute_raw(m, Lf, Lf);  // T_pf(L, 0) - T_pf(0, L)
      const float W0 = fmaxf(0.0f, Z);
      const uint32_t n0 = nA - nCand;
      uint32_t wmin_bits = n0 > 0 ? __float_as_uint(W0) : 0x7F800000u;
      if (few) {
        if ((uint32_t)lane < nCand) {
          const float W = fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)myhit * m.bs), Lf));
          const uint32_t wb = __float_as_uint(W);
          wmin_bits = wb < wmin_bits ? wb : wmin_bits;
        }
      } else {
        for (int32_t base = 0; base < n_inst; base += 64) {
          const int32_t i = base + lane;
          const bool cand = i < n_inst && test_bit(bmC, (uint32_t)i);
          uint32_t v = cand ? hits[i] : 0u;
          uint64_t ovf = __ballot(cand && v == kHitOverflow);
          while (ovf) {  // hits beyond the u16 slot: walk again
            const int k = __builtin_ctzll(ovf);
            ovf &= ovf - 1;
            const uint32_t hk =
                grp ? run_walk<false>(a.t, (uint32_t)(base + k), c, nullptr, 0, g, s)
                    : run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
            if (lane == k) v = hk;
          }
          if (cand) {
            const float W = fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)v * m.bs), Lf));
            const uint32_t wb = __float_as_uint(W);
            wmin_bits = wb < wmin_bits ? wb : wmin_bits;
          }
        }
      }
      const float wmin = __uint_as_float(wave_min_u32(wmin_bits));

      // (3)-(4) Filters and keys.  The hit-0 class is visited only if its
      // common penalty passes Eq. 9.
      const float tpf_cold = t_prefill(m, Lf, 0.0f);
      const float slo = fmaxf(m.ttft_floor, tpf_cold);
      const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
      const bool admit0 = n0 > 0 && (!kvc || (W0 - wmin) / Z <= m.eta);
      Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
      if (nA > 0) {
        if (few) {
          if ((uint32_t)lane < nCand)
            evaluate_with<FAST>(m, acc, myid, myhit, [&]() { return state_of(myid); }, L, Lf, wmin, Z, kvc,
                          slo);
        } else {
          for (int32_t base = 0; base < n_inst; base += 64) {
            const int32_t i = base + lane;
            const bool cand = i < n_inst && test_bit(bmC, (uint32_t)i);
            uint32_t v = cand ? hits[i] : 0u;
            uint64_t ovf = __ballot(cand && v == kHitOverflow);
            while (ovf) {
              const int k = __builtin_ctzll(ovf);
              ovf &= ovf - 1;
              const uint32_t hk =
                  grp ? run_walk<false>(a.t, (uint32_t)(base + k), c, nullptr, 0, g, s)
                      : run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
              if (lane == k) v = hk;
            }
            if (cand)
              evaluate_with<FAST>(m, acc, (uint32_t)i, v, [&]() { return state_of((uint32_t)i); }, L, Lf,
                            wmin, Z, kvc, slo);
          }
        }
        if (admit0) {
          // The eligible non-holders (hit 0) share n = L.  Without set sizes
          // to report, only the best packing key of that class matters: the
          // first member of T in key order (decoding desc, queued asc, id
          // asc).  The whole class is evaluated when sizes are requested or
          // when no member is in T (then the fallback key may come from it).
          bool done0 = false, searched = false;
          const bool keyed = FAST || m.sel == PS_SEL_DCQ || m.sel == PS_SEL_DQ || m.sel == PS_SEL_DQC;
          if (!sizes && keyed && (FAST || (m.mono && !(m.flags & PS_F_TTFT_ADMIT)))) {
            searched = true;
            // The first member of T in key order: the first key position whose
            // threshold admits this length and whose instance does not hold
            // the first block.  Chunk maxima skip 64 positions per entry.
            const int32_t n1 = (n_inst + 63) >> 6;
            for (int32_t c0 = 0; c0 < n1 && !done0; c0 += 64) {
              const int32_t cc = c0 + lane;
              uint64_t cm = __ballot(cc < n1 && (SMALL || (FAST ? llm1v[cc] : a.lm1[cc]) >= ell));
              while (cm && !done0) {
                const int32_t k0 = (c0 + __builtin_ctzll(cm)) * 64;
                cm &= cm - 1;
                const int32_t k = k0 + lane;
                const int4 e = k < n_inst ? (SMALL ? llm[k] : a.lm[k]) : make_int4(-1, 0, 0, 0);
                const uint64_t om = __ballot(e.x >= ell && !test_bit(bmC, (uint32_t)e.y));
                if (om) {
                  if (lane == __builtin_ctzll(om)) {
                    InstState st{};
                    st.D = e.z;
                    st.Q = e.w;
                    const uint64_t kt = select_key(m.sel, st, 0u, (uint32_t)e.y, 0ull);
                    acc.keyT = kt < acc.keyT ? kt : acc.keyT;
                  }
                  done0 = true;
                }
              }
            }
          } else if (!sizes && keyed) {
            searched = true;
            for (int32_t base = 0; base < n_inst && !done0; base += 64) {
              const int32_t k = base + lane;
              bool ok = false;
              uint32_t i = 0;
              InstState st{};
              if (k < n_inst) {
                i = a.order0[k];
                st = a.inst_key[k];  // contiguous, loaded with the id
                if (eligible(m, st.A1, st.S, L) && !test_bit(bmC, i)) {
                  const Lat lt = latency(m, st, Lf, 0.0f, L);
                  ok = ((m.flags & PS_F_NO_TPOT_FILTER) || lt.tpot < m.tau) &&
                       (!(m.flags & PS_F_TTFT_ADMIT) || lt.ttft <= slo);
                }
              }
              const uint64_t okm = __ballot(ok);
              if (okm) {
                if (lane == __builtin_ctzll(okm)) {
                  const uint64_t kt = select_key(m.sel, st, 0u, i, 0ull);
                  acc.keyT = kt < acc.keyT ? kt : acc.keyT;
                }
                done0 = true;
              }
            }
          }
          // A search found no member of the class in T: its keys matter only
          // for the fallback, i.e. when no candidate is in T either.
          if (!done0 && searched) done0 = wave_min_u64(acc.keyT) != ~0ull;
          if (!done0) {
            for (int32_t base = 0; base < n_inst; base += 64) {
              const int32_t i = base + lane;
              if (i < n_inst && !test_bit(bmC, (uint32_t)i) && room_of((uint32_t)i) >= L)
                evaluate_with<FAST>(m, acc, (uint32_t)i, 0u, [&]() { return state_of((uint32_t)i); }, L, Lf,
                              wmin, Z, kvc, slo);
            }
          }
        }
      }
      uint64_t keyT;
      if (sel_hcq) {  // smallest headroom first, then the rest of the key
        const uint64_t hmin = wave_min_u64((uint64_t)acc.hroom);
        keyT = wave_min_u64((uint64_t)acc.hroom == hmin ? acc.keyT : ~0ull);
      } else {
        keyT = wave_min_u64(acc.keyT);
      }
      // the fallback key matters only when T is empty; the set sizes only
      // when reported or for the random selector
      const uint64_t keyF = keyT == ~0ull ? wave_min_u64(acc.keyF) : ~0ull;
      const bool counts = sizes || sel_random;
      const uint32_t nC = counts ? wave_sum_u32(acc.nC) : 0u;
      const uint32_t nT = counts ? wave_sum_u32(acc.nT) : 0u;
      if (sel_random && nT > 0) {
        // the k-th member of T in id order
        const uint64_t z = splitmix64_at(m.rand_seed, r);
        const uint32_t kth = (uint32_t)(((z >> 32) * (uint64_t)nT) >> 32);
        uint32_t seen = 0;
        for (int32_t base = 0; base < n_inst; base += 64) {
          const int32_t i = base + lane;
          const bool el = i < n_inst && room_of((uint32_t)i) >= L;
          const bool cand = el && test_bit(bmC, (uint32_t)i);
          uint32_t v = cand ? hits[i] : 0u;
          uint64_t ovf = __ballot(cand && v == kHitOverflow);
          while (ovf) {
            const int k = __builtin_ctzll(ovf);
            ovf &= ovf - 1;
            const uint32_t hk = grp ? run_walk<false>(a.t, (uint32_t)(base + k), c, nullptr, 0, g, s)
                                    : run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
            if (lane == k) v = hk;
          }
          bool inT = false;
          if (el && (cand || admit0))
            inT = member_with<FAST>(m, [&]() { return state_of((uint32_t)i); }, v, L, Lf, wmin, Z, kvc, slo)
                      .inT;
          uint64_t mm = __ballot(inT);
          const uint32_t cnt = (uint32_t)__popcll(mm);
          if (seen + cnt > kth) {
            for (uint32_t j = seen; j < kth; ++j) mm &= mm - 1;
            keyT = (uint64_t)(base + __builtin_ctzll(mm));
            break;
          }
          seen += cnt;
        }
      }

      // Decision.  With finite arithmetic C holds at least the minimum-penalty
      // candidate whenever A is non-empty; the key test only keeps a
      // non-finite model from selecting an out-of-range id.
      ps_result res{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
      if (nA > 0 && (keyT != ~0ull || keyF != ~0ull)) {
        uint32_t fl = 0;
        uint32_t best;
        if (keyT != ~0ull) {
          best = (uint32_t)(keyT & 0xFFFFu);
        } else {
          best = (uint32_t)(keyF & 0xFFFFu);
          fl |= PS_R_FALLBACK;
        }
        uint32_t v = 0;
        if (test_bit(bmC, best)) {
          if (few) {
            const uint64_t mk = __ballot((uint32_t)lane < nCand && myid == best);
            v = (uint32_t)__shfl((int)myhit, __builtin_ctzll(mk));
          } else {
            v = hits[best];
            if (v == kHitOverflow)
              v = grp ? run_walk<false>(a.t, best, c, nullptr, 0, g, s)
                      : run_walk<true>(a.t, best, c, stage, 0, g, s);
          }
        }
        const int64_t c_tok = (int64_t)v * m.bs;
        const InstState st = state_of(best);
        const Lat lt = latency(m, st, (float)(L - c_tok), (float)c_tok, L);
        if (lt.ttft > slo) fl |= PS_R_TTFT_MISS;
        res = ps_result{(int32_t)best, (int32_t)v, lt.ttft, lt.tpot, fl};
      }
      if (lane == 0) {
        a.out[r] = res;
        if (sizes) {
          sizes[3 * (size_t)r] = nA;
          sizes[3 * (size_t)r + 1] = nC;
          sizes[3 * (size_t)r + 2] = nT;
        }
      }
      // leave the candidate bitmap clear for the next request
      __syncthreads();
      if (few) {
        if ((uint32_t)lane < nCand) bmC[myid >> 6] = 0ull;
      } else {
        for (int32_t w = lane; w < nw; w += 64) bmC[w] = 0ull;
      }
    }
  }
}

// ------------------------------------------------------------ lean scorer
// Scoring of the requests whose group record holds their hits (at most
// kGroupHold holders of the first block), for every selector except Random
// and H-C-Q.  Its read schedule is built for a chain of dependent reads
// per request: a wave's batch of descriptors, slots and records arrive in
// two round trips; the pool's 64 largest rooms and the zero-hit threshold
// maxima (window constants) sit in registers for the whole launch; per
// request the holders' states (which also decide their eligibility) and
// the first passing chunk of zero-hit thresholds, with the key-ordered
// states, are read together, so a decision usually needs one more round
// trip after the record.  Every other valid request is marked kDeferred
// (and *a.defer_any set) for the general kernel that follows.
template <bool SMALL>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void lean_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int32_t n_inst = a.n_inst;
  const int32_t nw = (n_inst + 63) >> 6;
  uint64_t* bmH = reinterpret_cast<uint64_t*>(smem);  // holders of the request's first block
  uint2* lrec = reinterpret_cast<uint2*>(bmH + ((nw + 1) & ~1));
  int64_t* lq64 = reinterpret_cast<int64_t*>(lrec + kBatch * kGroupRec);
  uint32_t* lgso = reinterpret_cast<uint32_t*>(lq64 + 3 * kBatch);
  InstState* linst = reinterpret_cast<InstState*>(lgso + kBatch);  // SMALL: states by id
  int4* llm = reinterpret_cast<int4*>(linst + kSmallPool);          // SMALL: thresholds
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  __shared__ DevModel lmodel;  // visible after the barrier below
  stage_model(lmodel, a.model, lane, 64);
  const DevModel& m = lmodel;
  for (int32_t w = lane; w < nw; w += 64) bmH[w] = 0ull;
  const TopRoom trm = a.rtop[lane];
  const int32_t n1 = (n_inst + 63) >> 6;
  const int32_t lm1r = lane < n1 ? a.lm1[lane] : -1;
  if (SMALL && lane < n_inst) {
    linst[lane] = a.inst[lane];
    llm[lane] = a.lm[lane];
  }
  __syncthreads();
  auto state_of = [&](uint32_t i) -> InstState { return SMALL ? linst[i] : a.inst[i]; };
  const bool keyed = m.sel == PS_SEL_DCQ || m.sel == PS_SEL_DQ || m.sel == PS_SEL_DQC;
  const bool fast0 = !a.sizes && keyed && m.mono && !(m.flags & PS_F_TTFT_ADMIT);
  bool deferred_any = false;

  const int32_t B = a.batch;
  for (int32_t rb = blockIdx.x * B; rb < a.n_req; rb += gridDim.x * B) {
    const int32_t nb = a.n_req - rb < B ? a.n_req - rb : B;
    __syncthreads();  // the previous batch is done with the batch buffers
    if (lane < nb) lgso[lane] = a.grp.slot_of[rb + lane];
    if (lane < 3 * nb) lq64[lane] = reinterpret_cast<const int64_t*>(a.reqs + rb)[lane];
    __syncthreads();
    for (int32_t w = lane; w < nb * kGroupRec; w += 64) {
      const uint32_t so = lgso[w / kGroupRec];
      if (so != kGroupNoSlot)
        lrec[w] = a.grp.rec[(size_t)(so & ~kGroupLead) * kGroupRec + (uint32_t)(w % kGroupRec)];
    }
    __syncthreads();
    for (int32_t b = 0; b < nb; ++b) {
      const int32_t r = rb + b;
      const uint32_t gso = (uint32_t)__builtin_amdgcn_readfirstlane((int)lgso[b]);
      const ps_req ql = reinterpret_cast<const ps_req*>(lq64)[b];
      const ps_req q{uniform64(ql.pre_off), uniform64(ql.tail_off),
                     __builtin_amdgcn_readfirstlane(ql.pre_len),
                     __builtin_amdgcn_readfirstlane(ql.tail_len)};
      if (!req_valid(q, a.pool_len)) {
        if (lane == 0) {
          a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_INVALID};
          if (a.sizes) a.sizes[3 * (size_t)r] = a.sizes[3 * (size_t)r + 1] = a.sizes[3 * (size_t)r + 2] = 0;
        }
        continue;
      }
      uint32_t cnt = kGroupNone;
      uint2 hd = make_uint2(0u, 0u);
      if (gso != kGroupNoSlot) {
        const uint2* grec = lrec + b * kGroupRec;
        cnt = (uint32_t)__builtin_amdgcn_readfirstlane((int)grec[0].y);
        if ((uint32_t)lane < kGroupHold) hd = grec[1 + lane];
      }
      if (cnt == kGroupNone || (cnt & kGroupPop)) {  // no record with the hits: the general kernel
        if (lane == 0) a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, kDeferred};
        deferred_any = true;
        continue;
      }
      const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
      const int32_t ell = c.len;
      const int64_t L = (int64_t)ell * m.bs;
      const float Lf = (float)L;
      const int32_t p = q.pre_len;
      uint32_t nA_exact = 0;
      if (a.sizes) nA_exact = (uint32_t)(n_inst - wave_lower_bound(a.room_sorted, n_inst, L, lane));
      if (!(__shfl(trm.room, 0) >= L)) {  // A is empty: Reject
        if (lane == 0) {
          a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
          if (a.sizes) a.sizes[3 * (size_t)r] = a.sizes[3 * (size_t)r + 1] = a.sizes[3 * (size_t)r + 2] = 0;
        }
        continue;
      }
      // The first chunk of zero-hit thresholds that admits this length, with
      // the key-ordered states, read together with the holders' states.
      uint64_t cmask = fast0 ? __ballot(lane < n1 && lm1r >= ell) : 0ull;
      int32_t c0 = 0;
      int4 e = make_int4(-1, 0, 0, 0);
      InstState est{};
      bool have = false;
      if (cmask) {
        const int32_t k = (int32_t)__builtin_ctzll(cmask) * 64 + lane;
        if (k < n_inst) {
          e = SMALL ? llm[k] : a.lm[k];
          if (!SMALL) est = a.inst_key[k];
        }
        have = true;
      }
      // Holders: state (and with it eligibility) and hit; the holder bitmap.
      InstState hst{};
      bool el = false;
      uint32_t id = 0, hit = 0;
      if ((uint32_t)lane < cnt) {
        id = hd.x;
        hit = hd.y;
        hst = state_of(id);
        el = eligible(m, hst.A1, hst.S, L);
        atomicOr(reinterpret_cast<unsigned long long*>(&bmH[id >> 6]), 1ull << (id & 63));
      }
      if (SMALL && have && e.x >= 0) est = linst[e.y];
      __syncthreads();
      // Hits that reach the request's segment end continue on its tail.
      uint64_t need = __ballot(el && (int32_t)hit >= p);
      while (need) {
        const int k = __builtin_ctzll(need);
        need &= need - 1;
        const uint32_t idk = (uint32_t)__shfl((int)id, k);
        const uint32_t hk = run_walk<false>(a.t, idk, c, nullptr, p, g, s);
        if (lane == k) hit = hk;
      }
      // Some eligible instance holds nothing (exact from the 64 largest
      // rooms: 64 eligible ones cannot all be among at most 16 holders).
      const bool topel = trm.room >= L;
      const bool any0 = __ballot(topel && !test_bit(bmH, (uint32_t)trm.id)) != 0ull ||
                        __shfl(topel ? 1 : 0, 63) != 0;
      // Minimum recomputation penalty over A.
      const float Z = recompute_raw(m, Lf, Lf);  // T_pf(L, 0) - T_pf(0, L)
      const float W0 = fmaxf(0.0f, Z);
      uint32_t wb = 0x7F800000u;
      if (el) wb = __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)hit * m.bs), Lf)));
      if (any0 && lane == 0) wb = wb < __float_as_uint(W0) ? wb : __float_as_uint(W0);
      const float wmin = __uint_as_float(wave_min_u32(wb));
      const float tpf_cold = t_prefill(m, Lf, 0.0f);
      const float slo = fmaxf(m.ttft_floor, tpf_cold);
      const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
      const bool admit0 = any0 && (!kvc || (W0 - wmin) / Z <= m.eta);
      Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
      if (el) evaluate_with(m, acc, id, hit, [&]() { return hst; }, L, Lf, wmin, Z, kvc, slo);
      // The hit-0 class: eligible non-holders, one penalty W(L).
      int32_t win0 = -1;  // lane of the class member found by the search
      if (admit0) {
        bool done0 = false;
        if (fast0) {
          while (have) {
            const uint64_t om = __ballot(e.x >= ell && !test_bit(bmH, (uint32_t)e.y));
            if (om) {
              win0 = __builtin_ctzll(om);
              if (lane == win0) {
                InstState kst{};
                kst.D = e.z;
                kst.Q = e.w;
                const uint64_t kt = select_key(m.sel, kst, 0u, (uint32_t)e.y, 0ull);
                acc.keyT = kt < acc.keyT ? kt : acc.keyT;
              }
              done0 = true;
              break;
            }
            // the next chunk whose maximum admits this length
            cmask &= cmask - 1;
            while (!cmask) {
              c0 += 64;
              if (c0 >= n1) break;
              const int32_t cc = c0 + lane;
              cmask = __ballot(cc < n1 && a.lm1[cc] >= ell);
            }
            have = cmask != 0ull;
            if (have) {
              const int32_t k = (c0 + (int32_t)__builtin_ctzll(cmask)) * 64 + lane;
              e = make_int4(-1, 0, 0, 0);
              if (k < n_inst) {
                e = SMALL ? llm[k] : a.lm[k];
                est = SMALL ? linst[e.y] : a.inst_key[k];
              }
            }
          }
          // No member of the class is in T: its keys matter only for the
          // fallback, i.e. when no candidate is in T either.
          if (!done0) done0 = wave_min_u64(acc.keyT) != ~0ull;
        }
        if (!done0) {  // the whole class, lanes over the pool
          for (int32_t base = 0; base < n_inst; base += 64) {
            const int32_t i = base + lane;
            if (i < n_inst && !test_bit(bmH, (uint32_t)i)) {
              const InstState st = state_of((uint32_t)i);
              if (eligible(m, st.A1, st.S, L))
                evaluate_with(m, acc, (uint32_t)i, 0u, [&]() { return st; }, L, Lf, wmin, Z, kvc,
                              slo);
            }
          }
        }
      }
      const uint64_t keyT = wave_min_u64(acc.keyT);
      const uint64_t keyF = keyT == ~0ull ? wave_min_u64(acc.keyF) : ~0ull;
      uint32_t nC = 0, nT = 0;
      if (a.sizes) {
        nC = wave_sum_u32(acc.nC);
        nT = wave_sum_u32(acc.nT);
      }
      // Decision: the chosen instance's state from the lane that read it.
      ps_result res{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
      if (keyT != ~0ull || keyF != ~0ull) {
        const bool t = keyT != ~0ull;
        const uint32_t best = (uint32_t)((t ? keyT : keyF) & 0xFFFFu);
        const uint64_t hb = __ballot(el && id == best);
        InstState bs{};
        uint32_t v = 0;
        if (hb) {
          const int src = __builtin_ctzll(hb);
          bs = shfl_state(hst, src);
          v = (uint32_t)__shfl((int)hit, src);
        } else if (win0 >= 0 && (uint32_t)__shfl(e.y, win0) == best) {
          bs = shfl_state(est, win0);
        } else {
          bs = state_of(best);
        }
        const int64_t c_tok = (int64_t)v * m.bs;
        const Lat lt = latency(m, bs, (float)(L - c_tok), (float)c_tok, L);
        res = ps_result{(int32_t)best, (int32_t)v, lt.ttft, lt.tpot,
                        (t ? 0u : PS_R_FALLBACK) | (lt.ttft > slo ? PS_R_TTFT_MISS : 0u)};
      }
      if (lane == 0) {
        a.out[r] = res;
        if (a.sizes) {
          a.sizes[3 * (size_t)r] = nA_exact;
          a.sizes[3 * (size_t)r + 1] = nC;
          a.sizes[3 * (size_t)r + 2] = nT;
        }
      }
      __syncthreads();
      if ((uint32_t)lane < cnt) bmH[id >> 6] = 0ull;
      __syncthreads();
    }
  }
  if (deferred_any && lane == 0) *a.defer_any = 1u;  // (a plain store: every writer writes 1)
}

// ------------------------------------------------------- lean scorer, rows
// The lean scorer with four requests per wave, one per row of 16 lanes:
// lane t of a row takes holder t of its request's record (at most
// kGroupHold = 16) and entries t, t + 16, t + 32, t + 48 of a chunk of
// zero-hit thresholds, so one wave-wide instruction serves four requests.
// Row reductions are DPP shifts inside the row.  It serves the common case
// of the keyed selectors (D-C-Q, D-Q, D-Q-C) with a monotone model, no TTFT
// admission and no candidate-set sizes, on pools of at most 4,096
// instances.  When no candidate is in T while the zero-hit class is in C,
// the row scans the whole class for its fallback keys.

// Minimum over the 16 lanes of each row, in every lane of the row.
__device__ __forceinline__ uint32_t row_min_u32(uint32_t v) {
  min32_step<0x111, 0xF>(v);  // row_shr:1
  min32_step<0x112, 0xF>(v);  // row_shr:2
  min32_step<0x114, 0xF>(v);  // row_shr:4
  min32_step<0x118, 0xF>(v);  // row_shr:8
  return (uint32_t)__shfl((int)v, (int)((threadIdx.x & 48u) | 15u));
}

__device__ __forceinline__ uint64_t row_min_u64(uint64_t v) {
  min_step<0x111, 0xF>(v);
  min_step<0x112, 0xF>(v);
  min_step<0x114, 0xF>(v);
  min_step<0x118, 0xF>(v);
  const int src = (int)((threadIdx.x & 48u) | 15u);
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src);
  const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

// This lane's row's 16 bits of a ballot.
__device__ __forceinline__ uint32_t row_bits(uint64_t b) {
  return (uint32_t)(b >> (threadIdx.x & 48u)) & 0xFFFFu;
}

template <bool SMALL>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4))) void lean_rows_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int32_t n_inst = a.n_inst;
  const int32_t nw = (n_inst + 63) >> 6;
  const int32_t nwp = (nw + 1) & ~1;
  uint64_t* bmall = reinterpret_cast<uint64_t*>(smem);                      // 4 holder bitmaps
  TopRoom* ltop = reinterpret_cast<TopRoom*>(bmall + 4 * (size_t)nwp);        // the 64 largest rooms
  int32_t* llm1 = reinterpret_cast<int32_t*>(ltop + kTopRooms);              // threshold chunk maxima
  InstState* linst = reinterpret_cast<InstState*>(llm1 + 64);                // SMALL: states by id
  int4* llm = reinterpret_cast<int4*>(linst + kSmallPool);                    // SMALL: thresholds
  const int lane = threadIdx.x;
  const int q = lane >> 4, t = lane & 15;
  const int g = lane >> 3, s = lane & 7;
  __shared__ DevModel lmodel;  // read by every batch (visible after the barrier below)
  stage_model(lmodel, a.model, lane, 64);
  const DevModel& m = lmodel;
  uint64_t* bmH = bmall + (size_t)q * nwp;  // this row's request's holders
  for (int32_t w = lane; w < 4 * nwp; w += 64) bmall[w] = 0ull;
  // window constants in LDS (read again per request: registers are scarce)
  {
    const TopRoom tr = a.rtop[lane];
    ltop[lane] = tr;
  }
  const int32_t n1 = (n_inst + 63) >> 6;  // <= 64
  llm1[lane] = lane < n1 ? a.lm1[lane] : -1;
  if (SMALL && lane < n_inst) {
    linst[lane] = a.inst[lane];
    llm[lane] = a.lm[lane];
  }
  __syncthreads();
  const int64_t room0 = ltop[0].room;    // the largest room
  const int64_t room63 = ltop[63].room;  // the 64th largest
  auto state_of = [&](uint32_t i) -> InstState { return SMALL ? linst[i] : a.inst[i]; };
  bool deferred_any = false;
  // Descriptor and slot of the row's request (every lane of a row reads its
  // row's); the next batch's are read near the end of the batch before, as
  // vectors (register tuples the loads fill in place) and unconditionally
  // at a request clamped into the window (n_req >= 1 here): a branch around
  // them would end in register copies that wait for the loads.
  uint4 qa;
  uint2 qb;
  uint32_t gn;
  auto read_desc = [&](int32_t rq) {
    const int32_t rc = rq < a.n_req ? rq : a.n_req - 1;
    const char* d = reinterpret_cast<const char*>(a.reqs + rc);
    qa = *reinterpret_cast<const uint4*>(d);
    qb = *reinterpret_cast<const uint2*>(d + 16);
    gn = a.grp.slot_of[rc];
  };
  static_assert(sizeof(ps_req) == 24, "a descriptor is 16 + 8 bytes");
  read_desc((int32_t)blockIdx.x * 4 + q);
  // Hand-over to the general kernel: a batch's left requests (lanes t = 0
  // of their rows in hdm, their ids in hr) go to this wave's sub-list at
  // the place the count atomic returned (lane 0's hbase).
  uint64_t hdm = 0ull;
  uint32_t hbase = 0u;
  int32_t hr = 0;
  int32_t* const hlist = a.dlist ? a.dlist + (size_t)(blockIdx.x % kDeferLists) * (size_t)a.dcap : nullptr;
  auto hand_over = [&]() {
    if (hdm != 0ull) {
      const uint32_t b0 = (uint32_t)__shfl((int)hbase, 0);
      if ((hdm >> lane) & 1ull) hlist[b0 + (uint32_t)__popcll(hdm & ((1ull << lane) - 1ull))] = hr;
    }
  };

  for (int32_t rb = blockIdx.x * 4; rb < a.n_req; rb += gridDim.x * 4) {
    const int32_t r = rb + q;
    const bool inr = r < a.n_req;
    // descriptor and slot, then the record
    const ps_req qd = inr ? ps_req{(int64_t)(((uint64_t)qa.y << 32) | qa.x),
                                   (int64_t)(((uint64_t)qa.w << 32) | qa.z), (int32_t)qb.x, (int32_t)qb.y}
                          : ps_req{0, 0, 0, 0};
    const uint32_t gso = inr ? gn : kGroupNoSlot;
    const bool valid = inr && req_valid(qd, a.pool_len);
    uint32_t cnt = kGroupNone;
    uint2 hd = make_uint2(0u, 0u);
    if (valid && gso != kGroupNoSlot) {
      const uint2* grec = a.grp.rec + (size_t)(gso & ~kGroupLead) * kGroupRec;
      cnt = grec[0].y;
      hd = grec[1 + t];
    }
    const ChainRef c{a.pool + qd.pre_off, a.pool + qd.tail_off, qd.pre_len, qd.pre_len + qd.tail_len};
    const int32_t ell = c.len;
    const int64_t L = (int64_t)ell * m.bs;
    const float Lf = (float)L;
    const int32_t p = qd.pre_len;
    // 0 scored here, 1 invalid, 2 left to the general kernel, 3 rejected
    uint32_t fate = !inr ? 4u : !valid ? 1u : (cnt == kGroupNone || (cnt & kGroupPop)) ? 2u
                                   : !(room0 >= L) ? 3u : 0u;
    const bool live = fate == 0u;
    // the first chunk of zero-hit thresholds that admits this length
    uint64_t cm = 0ull;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t ek = __builtin_amdgcn_readlane(ell, 16 * k);
      const uint64_t b = __ballot(lane < n1 && llm1[lane] >= ek);
      if (q == k) cm = b;
    }
    if (!live) cm = 0ull;
    // entries t + 16 u of the chunk (kept in registers: no array escapes)
    int4 e0, e1, e2, e3;
#define PS_ROWS_LOAD_CHUNK(cmask)                                                  \
    do {                                                                           \
      const uint64_t cmk = (cmask);                                                \
      const int32_t k0 = cmk ? (int32_t)__builtin_ctzll(cmk) * 64 + t : n_inst;   \
      e0 = k0 < n_inst ? (SMALL ? llm[k0] : a.lm[k0]) : make_int4(-1, 0, 0, 0);   \
      e1 = k0 + 16 < n_inst ? (SMALL ? llm[k0 + 16] : a.lm[k0 + 16]) : make_int4(-1, 0, 0, 0); \
      e2 = k0 + 32 < n_inst ? (SMALL ? llm[k0 + 32] : a.lm[k0 + 32]) : make_int4(-1, 0, 0, 0); \
      e3 = k0 + 48 < n_inst ? (SMALL ? llm[k0 + 48] : a.lm[k0 + 48]) : make_int4(-1, 0, 0, 0); \
    } while (0)
    PS_ROWS_LOAD_CHUNK(cm);
    // holders: state (and with it eligibility) and hit; the row's bitmap
    InstState hst{};
    bool el = false;
    uint32_t id = 0, hit = 0;
    if (live && (uint32_t)t < cnt) {
      id = hd.x;
      hit = hd.y;
      hst = state_of(id);
      el = eligible(m, hst.A1, hst.S, L);
      atomicOr(reinterpret_cast<unsigned long long*>(&bmH[id >> 6]), 1ull << (id & 63));
    }
    __syncthreads();
    // hits that reach the request's segment end continue on its tail
    uint64_t need = __ballot(el && (int32_t)hit >= p);
    while (need) {
      const int k = __builtin_ctzll(need);
      need &= need - 1;
      const int kr = k & 48;
      const ps_req qk{lane_value64(qd.pre_off, kr), lane_value64(qd.tail_off, kr),
                      __builtin_amdgcn_readlane(qd.pre_len, kr), __builtin_amdgcn_readlane(qd.tail_len, kr)};
      const ChainRef ck{a.pool + qk.pre_off, a.pool + qk.tail_off, qk.pre_len, qk.pre_len + qk.tail_len};
      const uint32_t idk = (uint32_t)__builtin_amdgcn_readlane((int)id, k);
      const uint32_t hk = run_walk<false, 2, 2>(a.t, idk, ck, nullptr, qk.pre_len, g, s);
      if (lane == k) hit = hk;
    }
    // some eligible instance holds nothing (exact from the 64 largest rooms:
    // 64 eligible ones cannot all be among at most 16 holders)
    bool any0 = false;
    {
      const TopRoom trm = ltop[lane];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t Lk = lane_value64(L, 16 * k);
        const uint64_t* bmk = bmall + (size_t)k * nwp;
        const bool ok = __ballot(trm.room >= Lk && !test_bit(bmk, (uint32_t)trm.id)) != 0ull || room63 >= Lk;
        if (q == k) any0 = ok;
      }
    }
    // minimum recomputation penalty over A
    const float Z = recompute_raw(m, Lf, Lf);  // T_pf(L, 0) - T_pf(0, L)
    const float W0 = fmaxf(0.0f, Z);
    uint32_t wb = 0x7F800000u;
    if (el) wb = __float_as_uint(fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)hit * m.bs), Lf)));
    if (any0 && t == 0) wb = wb < __float_as_uint(W0) ? wb : __float_as_uint(W0);
    const float wmin = __uint_as_float(row_min_u32(wb));
    const float tpf_cold = t_prefill(m, Lf, 0.0f);
    const float slo = fmaxf(m.ttft_floor, tpf_cold);
    const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
    const bool admit0 = live && any0 && (!kvc || (W0 - wmin) / Z <= m.eta);
    Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
    if (el) evaluate_with<true>(m, acc, id, hit, [&]() { return hst; }, L, Lf, wmin, Z, kvc, slo);
    // the hit-0 class: eligible non-holders, one penalty W(L); its first
    // admitted member in key order
    bool searching = admit0 && cm != 0ull;
    bool found0 = false;
    while (__ballot(searching) != 0ull) {
      uint32_t jmin = 64u;
      {
        const uint32_t f3 = row_bits(__ballot(searching && e3.x >= ell && !test_bit(bmH, (uint32_t)e3.y)));
        const uint32_t f2 = row_bits(__ballot(searching && e2.x >= ell && !test_bit(bmH, (uint32_t)e2.y)));
        const uint32_t f1 = row_bits(__ballot(searching && e1.x >= ell && !test_bit(bmH, (uint32_t)e1.y)));
        const uint32_t f0 = row_bits(__ballot(searching && e0.x >= ell && !test_bit(bmH, (uint32_t)e0.y)));
        if (f3) jmin = 48u + (uint32_t)__builtin_ctz(f3);
        if (f2) jmin = 32u + (uint32_t)__builtin_ctz(f2);
        if (f1) jmin = 16u + (uint32_t)__builtin_ctz(f1);
        if (f0) jmin = (uint32_t)__builtin_ctz(f0);
      }
      if (searching && jmin < 64u) {
        searching = false;
        found0 = true;
        if ((uint32_t)t == (jmin & 15u)) {
          const uint32_t uw = jmin >> 4;
          const int4 ew = uw == 0 ? e0 : uw == 1 ? e1 : uw == 2 ? e2 : e3;
          InstState kst{};
          kst.D = ew.z;
          kst.Q = ew.w;
          const uint64_t kt = select_key(m.sel, kst, 0u, (uint32_t)ew.y, 0ull);
          acc.keyT = kt < acc.keyT ? kt : acc.keyT;
        }
      } else if (searching) {  // the next chunk whose maximum admits this length
        cm &= cm - 1;
        searching = cm != 0ull;
      }
      if (__ballot(searching) == 0ull) break;  // (no row loads another chunk)
      PS_ROWS_LOAD_CHUNK(searching ? cm : 0ull);
    }
#undef PS_ROWS_LOAD_CHUNK
    uint64_t keyT = row_min_u64(acc.keyT);
    // no candidate in T while the class is in C: its fallback keys need the
    // whole class (16 lanes over the pool)
    const bool scan = live && keyT == ~0ull && admit0 && !found0;
    if (__ballot(scan) != 0ull) {
      for (int32_t base = 0; base < n_inst; base += 16) {
        const int32_t i = base + t;
        if (scan && i < n_inst && !test_bit(bmH, (uint32_t)i)) {
          const InstState st = state_of((uint32_t)i);
          if (eligible(m, st.A1, st.S, L))
            evaluate_with<true>(m, acc, (uint32_t)i, 0u, [&]() { return st; }, L, Lf, wmin, Z, kvc, slo);
        }
      }
      keyT = row_min_u64(acc.keyT);
    }
    const uint64_t kF = row_min_u64(acc.keyF);
    const uint64_t keyF = keyT == ~0ull ? kF : ~0ull;
    ps_result res{-1, 0, 0.0f, 0.0f, PS_R_REJECT};
    const bool chosen = fate == 0u && (keyT != ~0ull || keyF != ~0ull);
    const bool tt = keyT != ~0ull;
    const uint32_t best = (uint32_t)((tt ? keyT : keyF) & 0xFFFFu);
    // the chosen instance's state is read again (keeping the holders'
    // states live to here would spill)
    InstState bs{};
    if (chosen) bs = state_of(best);
    // the next batch's descriptors and slots, issued after this batch's last
    // read: vector loads return in order, so issued earlier these (usually
    // HBM misses) would hold up this batch's waits for its own L2 hits (an
    // earlier variant that read them at the start of the batch was 124 ->
    // 131 us at 4,096 x 262,144; this one 107 -> 105 us)
    __builtin_amdgcn_sched_barrier(0);
    {
      read_desc(rb + (int32_t)gridDim.x * 4 + q);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (chosen) {
      // its hit from the holder's lane
      const uint32_t hb = row_bits(__ballot(el && id == best));
      const int src = (lane & 48) + (hb ? __builtin_ctz(hb) : 0);
      const uint32_t sv = (uint32_t)__shfl((int)hit, src);
      const uint32_t v = hb ? sv : 0u;
      const int64_t c_tok = (int64_t)v * m.bs;
      const Lat lt = latency(m, bs, (float)(L - c_tok), (float)c_tok, L);
      res = ps_result{(int32_t)best, (int32_t)v, lt.ttft, lt.tpot,
                      (tt ? 0u : PS_R_FALLBACK) | (lt.ttft > slo ? PS_R_TTFT_MISS : 0u)};
    }
    if (t == 0 && fate != 4u) {
      if (fate == 1u) a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_INVALID};
      else if (fate == 2u) a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, kDeferred};
      else a.out[r] = res;
    }
    if (fate == 2u) deferred_any = true;
    if (a.dlist) {
      // the previous batch's left requests: their positions have arrived
      hand_over();
      // this batch's: places reserved now, written a batch later (the
      // count atomic's return is not waited for here)
      hdm = __ballot(t == 0 && fate == 2u);
      hr = r;
      if (hdm != 0ull && lane == 0)
        hbase = atomicAdd(a.dcnt + (blockIdx.x % kDeferLists) * kDeferStride, (uint32_t)__popcll(hdm));
    }
    __syncthreads();
    if (live && (uint32_t)t < cnt) bmH[id >> 6] = 0ull;
    __syncthreads();
  }
  if (a.dlist) hand_over();
  if (__ballot(deferred_any) != 0ull && lane == 0) *a.defer_any = 1u;  // (a plain store: every writer writes 1)
}

// One wave per instance that receives placements; its entries are applied
// in array order, each measured against the table as the earlier entries
// left it.
__global__ __launch_bounds__(64) void commit_kernel(CommitArgs a) {
  const int32_t g = blockIdx.x;
  const int lane = threadIdx.x;
  const uint32_t inst = (uint32_t)a.grp_inst[g];
  const DevModel& m = *a.model;
  InstState st = a.inst[inst];
  uint32_t count = a.t.count[inst];
  unsigned long long dropped = 0;
  for (int32_t k = a.grp_off[g]; k < a.grp_off[g + 1]; ++k) {
    const ps_req q = a.reqs[a.order[k]];
    const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
    const int32_t ell = c.len;
    const int64_t L = (int64_t)ell * m.bs;
    const uint32_t h = deep_walk<false>(a.t, inst, c, nullptr, 0, lane >> 3, lane & 7);
    st.Q += 1;
    st.A1 += 1;
    st.P += L - (int64_t)h * m.bs;
    st.S += L;
    for (int32_t base = 0; base < ell; base += 64) {
      const int32_t j = base + lane;
      const bool in = j < ell;
      const uint64_t key = in ? chain_global(c, j) : 0ull;
      const bool present = in ? probe(a.t, inst, key) : true;
      // repeated keys inside this chunk: only the first occurrence counts
      int first = lane;
      for (int s = 63; s >= 0; --s) {
        const uint64_t o = __shfl(key, s);
        if (s < lane && o == key) first = s;
      }
      const bool dup = first != lane;
      const bool want = in && !present && !dup;
      const uint64_t wm = __ballot(want);
      const uint32_t rank = (uint32_t)__popcll(wm & ((1ull << lane) - 1ull));
      const uint32_t room = a.cap > count ? a.cap - count : 0u;
      const bool ins = want && rank < room;
      if (ins) {  // new blocks join the row in chain order
        uint32_t slot = 0;
        (void)insert_key(a.t, inst, key, &slot);
        a.t.rows[(size_t)inst * a.t.row_cap + count + rank] = key;
        a.t.rowpos[(size_t)inst * a.t.slots + slot] = count + rank;
      }
      const uint64_t im = __ballot(ins);
      const uint64_t dup_drop = __ballot(in && dup && !present && !((im >> first) & 1ull));
      const uint32_t nins = (uint32_t)__popcll(im);
      count += nins;
      dropped += (unsigned long long)(__popcll(wm) - nins + __popcll(dup_drop));
      // later probes of this wave must see these inserts (workgroup scope: a
      // device-scope fence would write back the XCD's whole L2)
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    }
  }
  st.seg = segment_of(m, st.A1);
  if (lane == 0) {
    a.inst[inst] = st;
    a.room[inst] = st.A1 <= m.b_max ? m.kv_cap - st.S : -1;
    a.t.count[inst] = count;
    if (dropped) atomicAdd(a.dropped, dropped);
  }
}

}  // namespace

// ------------------------------------------------------------------ launchers
bool ps_score_small(int32_t n_inst) { return n_inst <= kSmallPool; }

int32_t ps_score_batch(int32_t n_req, int32_t resident_waves) {
  const int32_t b = resident_waves > 0 ? n_req / resident_waves : 1;
  return b < 1 ? 1 : (b > kBatch ? kBatch : b);
}

size_t ps_score_lds_bytes(int32_t n_inst) {
  return score_lds_base(n_inst, ps_hits_fit_lds(n_inst)) + kBatchLds +
         (ps_score_small(n_inst)
              ? (size_t)kSmallPool * (sizeof(int64_t) + sizeof(InstState) + sizeof(int4))
              : 0);
}

bool ps_hits_fit_lds(int32_t n_inst) {
  return (size_t)n_inst * sizeof(uint16_t) <= kLdsHitBudget;
}

hipError_t ps_launch_build(const BuildArgs& a, hipStream_t s) {
  if (a.n_blk == 0) return hipSuccess;
  int64_t blocks = (a.n_blk + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(build_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t ps_launch_rows(const BuildArgs& a, hipStream_t s) {
  if (a.n_blk == 0) return hipSuccess;
  int64_t blocks = (a.n_blk + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(row_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

size_t ps_lean_lds_bytes(int32_t n_inst) {
  const size_t nw = ((size_t)n_inst + 63) / 64;
  return ((nw + 1) & ~(size_t)1) * sizeof(uint64_t) + (size_t)kBatch * kGroupRec * sizeof(uint2) +
         3 * (size_t)kBatch * sizeof(int64_t) + (size_t)kBatch * sizeof(uint32_t) +
         (ps_score_small(n_inst) ? (size_t)kSmallPool * (sizeof(InstState) + sizeof(int4)) : 0);
}

int32_t ps_lean_waves_per_cu(int32_t n_inst) {
  int blocks = 0;
  const size_t lds = ps_lean_lds_bytes(n_inst);
  const hipError_t e =
      ps_score_small(n_inst)
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, lean_kernel<true>, 64, lds)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, lean_kernel<false>, 64, lds);
  return e == hipSuccess && blocks > 0 ? blocks : 16;
}

hipError_t ps_launch_score(const ScoreArgs& a, bool hits_in_lds, int grid, bool probe_all,
                           hipStream_t s, bool fast) {
  if (a.n_req == 0) return hipSuccess;
  if (probe_all) {
    // two 64-instance steps of first-block probes and 128 walk positions
    // in flight per wave (4 waves per SIMD)
    hipLaunchKernelGGL((probe_all_kernel<2, 2>), dim3(grid), dim3(64), (size_t)kStage * sizeof(uint64_t),
                       s, a);
    return hipGetLastError();
  }
  const size_t lds = ps_score_lds_bytes(a.n_inst);
  if (fast) {
    if (ps_score_small(a.n_inst))
      hipLaunchKernelGGL((score_kernel<true, true, true>), dim3(grid), dim3(64), lds, s, a);
    else if (hits_in_lds)
      hipLaunchKernelGGL((score_kernel<true, false, true>), dim3(grid), dim3(64), lds, s, a);
    else
      hipLaunchKernelGGL((score_kernel<false, false, true>), dim3(grid), dim3(64), lds, s, a);
  } else if (ps_score_small(a.n_inst)) {
    hipLaunchKernelGGL((score_kernel<true, true, false>), dim3(grid), dim3(64), lds, s, a);
  } else if (hits_in_lds) {
    hipLaunchKernelGGL((score_kernel<true, false, false>), dim3(grid), dim3(64), lds, s, a);
  } else {
    hipLaunchKernelGGL((score_kernel<false, false, false>), dim3(grid), dim3(64), lds, s, a);
  }
  return hipGetLastError();
}

hipError_t ps_launch_order(const ps_req* reqs, int32_t n, int64_t pool_len, uint32_t* bins,
                           int32_t* order, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int blocks = (n + 255) / 256;
  hipLaunchKernelGGL(order_clear_kernel, dim3(1), dim3(1024), 0, s, bins);
  hipLaunchKernelGGL(order_count_kernel, dim3(blocks), dim3(256), 0, s, reqs, n, pool_len, bins);
  hipLaunchKernelGGL(order_scan_kernel, dim3(1), dim3(1024), 0, s, bins);
  hipLaunchKernelGGL(order_place_kernel, dim3(blocks), dim3(256), 0, s, reqs, n, pool_len, bins,
                     order);
  return hipGetLastError();
}

hipError_t ps_launch_lean(const ScoreArgs& a, int grid, hipStream_t s) {
  if (a.n_req == 0) return hipSuccess;
  const size_t lds = ps_lean_lds_bytes(a.n_inst);
  if (ps_score_small(a.n_inst))
    hipLaunchKernelGGL(lean_kernel<true>, dim3(grid), dim3(64), lds, s, a);
  else
    hipLaunchKernelGGL(lean_kernel<false>, dim3(grid), dim3(64), lds, s, a);
  return hipGetLastError();
}

size_t ps_lean_rows_lds_bytes(int32_t n_inst) {
  const size_t nw = ((size_t)n_inst + 63) / 64;
  return 4 * ((nw + 1) & ~(size_t)1) * sizeof(uint64_t) + kTopRooms * sizeof(TopRoom) +
         64 * sizeof(int32_t) +
         (ps_score_small(n_inst) ? (size_t)kSmallPool * (sizeof(InstState) + sizeof(int4)) : 0);
}

int32_t ps_lean_rows_waves_per_cu(int32_t n_inst) {
  int blocks = 0;
  const size_t lds = ps_lean_rows_lds_bytes(n_inst);
  const hipError_t e =
      ps_score_small(n_inst)
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, lean_rows_kernel<true>, 64, lds)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, lean_rows_kernel<false>, 64, lds);
  return e == hipSuccess && blocks > 0 ? blocks : 16;
}

hipError_t ps_launch_lean_rows(const ScoreArgs& a, int grid, hipStream_t s) {
  if (a.n_req == 0) return hipSuccess;
  const size_t lds = ps_lean_rows_lds_bytes(a.n_inst);
  if (ps_score_small(a.n_inst))
    hipLaunchKernelGGL(lean_rows_kernel<true>, dim3(grid), dim3(64), lds, s, a);
  else
    hipLaunchKernelGGL(lean_rows_kernel<false>, dim3(grid), dim3(64), lds, s, a);
  return hipGetLastError();
}

int32_t ps_score_waves_per_cu(int32_t n_inst, bool hits_in_lds, bool fast) {
  int blocks = 0;
  const size_t lds = ps_score_lds_bytes(n_inst);
  hipError_t e;
  if (ps_score_small(n_inst))
    e = fast ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<true, true, true>, 64, lds)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<true, true, false>, 64, lds);
  else if (hits_in_lds)
    e = fast ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<true, false, true>, 64, lds)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<true, false, false>, 64, lds);
  else
    e = fast ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<false, false, true>, 64, lds)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, score_kernel<false, false, false>, 64, lds);
  return e == hipSuccess && blocks > 0 ? blocks : 12;
}

hipError_t ps_launch_lmax(const InstState* inst_key, const uint32_t* order0, const DevModel* m,
                          int32_t n, int4* lm, int32_t* lm1, uint4* csum, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(lmax_kernel, dim3((n + 63) / 64), dim3(64), 0, s, inst_key, order0, m, n, lm,
                     lm1, csum);
  return hipGetLastError();
}

hipError_t ps_launch_group(const ScoreArgs& a, int grid, hipStream_t s, hipEvent_t mid,
                           hipStream_t aux, hipEvent_t fork, hipEvent_t join) {
  if (a.n_req == 0) return hipSuccess;
  hipLaunchKernelGGL(group_claim_kernel, dim3((a.n_req + kClaimBlock - 1) / kClaimBlock),
                     dim3(kClaimBlock), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (mid) {
    e = hipEventRecord(mid, s);
    if (e != hipSuccess) return e;
  }
  const size_t nw = ((size_t)a.n_inst + 63) / 64;
  const size_t lds = (size_t)kStage * sizeof(uint64_t) + 2 * nw * sizeof(uint64_t);
  if (!a.grp.pop_pass) {
    hipLaunchKernelGGL(group_kernel, dim3(grid), dim3(64), lds, s, a);
    return hipGetLastError();
  }
  // the walk pass on the second stream, forked after the claim pass (which
  // lists the popular groups); the popular pass, the longer chain of
  // dependent launches, stays on the calling stream, which then waits for
  // the walk pass (long done by then: no cross-queue wake-up on the path)
  if (!aux || !fork || !join) return hipErrorInvalidValue;
  if ((e = hipEventRecord(fork, s)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(aux, fork, 0)) != hipSuccess) return e;
  hipLaunchKernelGGL(group_kernel, dim3(grid), dim3(64), lds, aux, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = hipEventRecord(join, aux)) != hipSuccess) return e;
  hipLaunchKernelGGL(popular_prefix_kernel, dim3(kPopPrefixGrid), dim3(64 * kPrefixWaves), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(popular_member_kernel, dim3(kPopWalkGrid), dim3(64), lds, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return hipStreamWaitEvent(s, join, 0);
}

hipError_t ps_launch_commit(const CommitArgs& a, hipStream_t s) {
  if (a.n_grp == 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3(a.n_grp), dim3(64), 0, s, a);
  return hipGetLastError();
}
