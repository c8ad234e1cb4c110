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
//                       (breadth probe of the first block, then deep walks).
//   commit_kernel     - ordered placement of decisions, one wave per instance.
//
// The path does no dense contraction, so it uses no MFMA.

#include "ps_device.h"

using namespace ps;

namespace {

// ---------------------------------------------------------------- reductions
// DPP row shifts and row broadcasts (GFX9 encodings): after the six steps
// lane 63 holds the reduction over all 64 lanes.  Lanes whose DPP source is
// out of range keep `old`, which is the identity of the operation.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_src(uint32_t identity, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)identity, (int)v, CTRL, ROW_MASK, 0xF, false);
}

template <int CTRL, int RM>
__device__ __forceinline__ void min_step(uint64_t& v) {
  const uint32_t lo = dpp_src<CTRL, RM>(0xFFFFFFFFu, (uint32_t)v);
  const uint32_t hi = dpp_src<CTRL, RM>(0xFFFFFFFFu, (uint32_t)(v >> 32));
  const uint64_t t = ((uint64_t)hi << 32) | lo;
  v = t < v ? t : v;
}

template <int CTRL, int RM>
__device__ __forceinline__ void add_step(uint32_t& v) {
  v += dpp_src<CTRL, RM>(0u, v);
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  min_step<0x111, 0xF>(v);  // row_shr:1
  min_step<0x112, 0xF>(v);  // row_shr:2
  min_step<0x114, 0xF>(v);  // row_shr:4
  min_step<0x118, 0xF>(v);  // row_shr:8
  min_step<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  min_step<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
  add_step<0x111, 0xF>(v);
  add_step<0x112, 0xF>(v);
  add_step<0x114, 0xF>(v);
  add_step<0x118, 0xF>(v);
  add_step<0x142, 0xA>(v);
  add_step<0x143, 0xC>(v);
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Exclusive prefix sum of v over the lanes of the wave.
__device__ __forceinline__ uint32_t wave_exclusive_sum(uint32_t v, int lane) {
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)x, d);
    if (lane >= d) x += y;
  }
  return x - v;
}

// Index of the first element >= L of an ascending array, 64 candidates per
// step: lanes read 64 evenly spaced samples and a ballot narrows the range
// by 64x (two dependent reads for up to 4096 elements).
__device__ __forceinline__ int32_t wave_lower_bound(const int64_t* arr, int32_t n, int64_t L,
                                                    int lane) {
  int32_t lo = 0, hi = n;
  while (hi - lo > 64) {
    const int32_t stride = (hi - lo + 63) / 64;
    const int32_t idx = lo + (lane + 1) * stride - 1;
    const bool less = idx < hi && arr[idx] < L;
    const int32_t c = (int32_t)__popcll(__ballot(less));
    const int32_t nlo = lo + c * stride;
    hi = hi < nlo + stride ? hi : nlo + stride;
    lo = nlo;
  }
  const int32_t idx = lo + lane;
  const bool less = idx < hi && arr[idx] < L;
  return lo + (int32_t)__popcll(__ballot(less));
}

// ------------------------------------------------------------------- probing
// Octet probing: the 8 lanes of an octet (lanes 8g .. 8g+7) read the 8 slots
// of one 64-byte bucket, so every wave-wide load is 8 coalesced 64-byte
// segments, and two ballots decide all 8 probes of the instruction.

struct Bucket {
  uint64_t k[kSlotsPerBucket];
};

__device__ __forceinline__ const uint64_t* table_of(const Tables& t, uint32_t inst) {
  return t.keys + (size_t)inst * (size_t)t.slots;
}

// Status of the probe of `key` by the octet of this lane, from the slot
// value this lane read: 1 found, 0 absent (an empty slot ends the probe
// sequence), 2 full bucket without the key (the next bucket decides).
// Inactive octets, and the zero hash (never stored), report 0.  Every lane
// of the wave must execute this (two ballots).
__device__ __forceinline__ uint32_t octet_status(uint64_t val, uint64_t key, bool act, int g) {
  const uint64_t fm = __ballot(act && val == key);
  const uint64_t em = __ballot(act && val == 0ull);
  const uint32_t f = (uint32_t)(fm >> (8 * g)) & 0xFFu;
  const uint32_t e = (uint32_t)(em >> (8 * g)) & 0xFFu;
  if (!act || key == 0ull) return 0u;
  return f ? 1u : (e ? 0u : 2u);
}

// Linear probing past full buckets for the octets still at status 2 (rare
// at load factor <= 0.5).  Wave-uniform loop, bounded by the bucket count.
__device__ __forceinline__ uint32_t octet_resolve(const Tables& t, const uint64_t* tab, uint32_t b,
                                                  uint64_t key, uint32_t status, int s, int g) {
  for (uint32_t step = 1; step <= t.bmask; ++step) {
    const bool pend = status == 2u;
    if (__ballot(pend) == 0ull) break;
    b = (b + 1) & t.bmask;
    const uint64_t val = pend ? tab[(size_t)b * kSlotsPerBucket + s] : 0ull;
    const uint32_t st = octet_status(val, key, pend, g);
    if (pend) status = st;
  }
  return status;
}

// Octet lookup in the prefix index: octet g looks up key (if act); the
// result is valid in every lane of the octet.  Every lane of the wave must
// call it.  One 16-byte entry per lane, one 128-byte bucket per octet.
struct IdxHit {
  bool found;
  uint32_t off, cnt;
};

__device__ __forceinline__ IdxHit index_lookup(const GIndex& x, uint64_t key, bool act, int g,
                                               int s) {
  IdxHit h{false, 0u, 0u};
  bool pend = act && key != 0ull;
  uint32_t b = bucket_of(key, kIndexSalt, x.shift);
  for (uint32_t step = 0; step <= x.bmask; ++step) {
    if (__ballot(pend) == 0ull) break;
    IdxEntry e{0ull, 0u, 0u};
    if (pend) e = x.ent[(size_t)b * kSlotsPerBucket + s];
    const uint64_t fm = __ballot(pend && e.key == key);
    const uint64_t em = __ballot(pend && e.key == 0ull);
    const uint32_t f = (uint32_t)(fm >> (8 * g)) & 0xFFu;
    const uint32_t z = (uint32_t)(em >> (8 * g)) & 0xFFu;
    const int src = 8 * g + (f ? __builtin_ctz(f) : 0);
    const uint32_t off = __shfl(e.off, src);
    const uint32_t cnt = __shfl(e.cnt, src);
    if (pend) {
      if (f) {
        h.found = true;
        h.off = off;
        h.cnt = cnt;
        pend = false;
      } else if (z) {
        pend = false;
      } else {
        b = (b + 1) & x.bmask;
      }
    }
  }
  return h;
}

// Single-lane lookup (commit path only).
__device__ __forceinline__ Bucket load_bucket(const uint64_t* p) {
  const ulonglong2* q = reinterpret_cast<const ulonglong2*>(p);
  const ulonglong2 a = q[0], b = q[1], c = q[2], d = q[3];
  return Bucket{{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y}};
}

__device__ bool probe(const Tables& t, uint32_t inst, uint64_t key) {
  if (key == 0) return false;
  const uint64_t* tab = table_of(t, inst);
  uint32_t b = bucket_of(key, inst, t.shift);
  for (uint32_t step = 0; step <= t.bmask; ++step) {
    const Bucket bk = load_bucket(tab + (size_t)b * kSlotsPerBucket);
    bool f = false, e = false;
#pragma unroll
    for (int s = 0; s < kSlotsPerBucket; ++s) {
      f |= bk.k[s] == key;
      e |= bk.k[s] == 0;
    }
    if (f) return true;
    if (e) return false;
    b = (b + 1) & t.bmask;
  }
  return false;
}

// 1 inserted, 0 already present, -1 no free slot; *slot = the key's slot
// within the instance's table.  Safe under concurrent inserts: a slot only
// ever changes from 0 to a key, and every claim of an apparently empty slot
// goes through a 64-bit compare-and-swap whose result decides.
__device__ int insert_key(const Tables& t, uint32_t inst, uint64_t key, uint32_t* slot) {
  uint64_t* tab = t.keys + (size_t)inst * (size_t)t.slots;
  uint32_t b = bucket_of(key, inst, t.shift);
  for (uint32_t step = 0; step <= t.bmask; ++step) {
    uint64_t* bp = tab + (size_t)b * kSlotsPerBucket;
    const Bucket bk = load_bucket(bp);
    for (int s = 0; s < kSlotsPerBucket; ++s)
      if (bk.k[s] == key) {
        *slot = b * kSlotsPerBucket + s;
        return 0;
      }
    for (int s = 0; s < kSlotsPerBucket; ++s) {
      if (bk.k[s] != 0) continue;
      const unsigned long long old =
          atomicCAS(reinterpret_cast<unsigned long long*>(bp + s), 0ull, (unsigned long long)key);
      if (old == 0ull || old == key) {
        *slot = b * kSlotsPerBucket + s;
        return old == 0ull ? 1 : 0;
      }
    }
    b = (b + 1) & t.bmask;
  }
  return -1;
}

// --------------------------------------------------------------------- chain
struct ChainRef {
  const uint64_t* pre;
  const uint64_t* tail;
  int32_t pre_len;
  int32_t len;
};

__device__ __forceinline__ uint64_t chain_global(const ChainRef& c, int32_t j) {
  return j < c.pre_len ? c.pre[j] : c.tail[j - c.pre_len];
}

__device__ __forceinline__ bool req_valid(const ps_req& q, int64_t pool_len) {
  return q.pre_len >= 0 && q.tail_len >= 0 && q.pre_off >= 0 && q.tail_off >= 0 &&
         q.pre_off <= pool_len && q.tail_off <= pool_len &&
         (int64_t)q.pre_len <= pool_len - q.pre_off &&
         (int64_t)q.tail_len <= pool_len - q.tail_off &&
         (int64_t)q.pre_len + (int64_t)q.tail_len <= (int64_t)PS_MAX_CHAIN;
}

// Deep walk of one instance: octets over chain positions.  A step issues
// the bucket reads of kDeepRounds x 8 positions, then prefetches the next
// step's chain hashes, then evaluates in chain order and stops at the first
// absent position.  Positions below kStage read the LDS copy of the chain.
// Wave-uniform arguments; returns the hit.
template <bool STAGED>
__device__ uint32_t deep_walk(const Tables& t, uint32_t inst, const ChainRef& c,
                              const uint64_t* stage, int32_t pos, int g, int s) {
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, inst);
  uint64_t nk[kDeepRounds];
#pragma unroll
  for (int r = 0; r < kDeepRounds; ++r) {
    const int32_t j = pos + r * 8 + g;
    nk[r] = 0ull;
    if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
  }
  while (pos < ell) {
    uint64_t key[kDeepRounds], val[kDeepRounds];
    uint32_t b[kDeepRounds];
#pragma unroll
    for (int r = 0; r < kDeepRounds; ++r) {
      const int32_t j = pos + r * 8 + g;
      key[r] = nk[r];
      b[r] = bucket_of(key[r], inst, t.shift);
      val[r] = 0ull;
      if (j < ell && key[r] != 0ull) val[r] = tab[(size_t)b[r] * kSlotsPerBucket + s];
    }
    const int32_t next = pos + kDeepRounds * 8;
#pragma unroll
    for (int r = 0; r < kDeepRounds; ++r) {
      const int32_t j = next + r * 8 + g;
      nk[r] = 0ull;
      if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
    }
#pragma unroll
    for (int r = 0; r < kDeepRounds; ++r) {
      const int32_t j = pos + r * 8 + g;
      const bool act = j < ell;
      uint32_t st = octet_status(val[r], key[r], act, g);
      st = octet_resolve(t, tab, b[r], key[r], st, s, g);
      const uint64_t miss = __ballot(act && st == 0u && s == 0);
      if (miss) return (uint32_t)(pos + r * 8 + (__builtin_ctzll(miss) >> 3));
    }
    pos = next;
  }
  return (uint32_t)ell;
}

// Walk of one instance along its row: one octet probe finds the block at
// `pos` and its row position; the chain blocks after it are compared with
// the row entries after it, 256 per step (4 per lane, coalesced), and the
// first mismatch is probed again (it may begin another run of the row, e.g.
// after a shared system prompt).  A run shorter than 8 blocks hands the rest
// of the walk to the octet walk.  Wave-uniform arguments; returns the hit.
template <bool STAGED>
__device__ __forceinline__ uint32_t run_walk(const Tables& t, uint32_t inst, const ChainRef& c,
                             const uint64_t* stage, int32_t pos, int g, int s) {
  const int lane = g * 8 + s;
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, inst);
  const uint64_t* row = t.rows + (size_t)inst * (size_t)t.row_cap;
  const int64_t rlen = t.count[inst];
  while (pos < ell) {
    const uint64_t key = (STAGED && pos < kStage) ? stage[pos] : chain_global(c, pos);
    if (key == 0ull) return (uint32_t)pos;
    uint32_t b = bucket_of(key, inst, t.shift);
    int64_t rp = -1;
    bool decided = false;
    for (uint32_t step = 0; step <= t.bmask && !decided; ++step) {
      const uint64_t val = g == 0 ? tab[(size_t)b * kSlotsPerBucket + s] : 0ull;
      const uint64_t fm = __ballot(g == 0 && val == key) & 0xFFull;
      const uint64_t em = __ballot(g == 0 && val == 0ull) & 0xFFull;
      if (fm) {
        rp = t.rowpos[(size_t)inst * t.slots + (size_t)b * kSlotsPerBucket + __builtin_ctzll(fm)];
        decided = true;
      } else if (em) {
        decided = true;
      } else {
        b = (b + 1) & t.bmask;
      }
    }
    if (rp < 0) return (uint32_t)pos;
    const int32_t start = pos + 1;
    int32_t q = start;
    int64_t k = rp + 1;
    int32_t next = -1;
    while (next < 0) {
      bool mism[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int32_t j = q + 64 * u + lane;
        const int64_t kk = k + 64 * u + lane;
        const bool valid = j < ell;
        uint64_t cj = 0ull, rk = 0ull;
        if (valid) cj = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
        if (valid && kk < rlen) rk = row[kk];
        mism[u] = valid && (kk >= rlen || cj != rk);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint64_t mm = __ballot(mism[u]);
        if (next < 0 && mm) next = q + 64 * u + __builtin_ctzll(mm);
      }
      if (next < 0) {
        q += 256;
        k += 256;
        if (q >= ell) return (uint32_t)ell;
      }
    }
    if (next - start < 8) return deep_walk<STAGED>(t, inst, c, stage, next, g, s);
    pos = next;
  }
  return (uint32_t)ell;
}

// ------------------------------------------------------------- latency model
// Eq. 7 with the empirical C and C^2 terms: n new, c cached tokens.
__device__ __forceinline__ float t_prefill(const DevModel& m, float n, float c) {
  return m.a[0] + n * (m.a[1] + m.a[2] * c + m.a[3] * n) + c * (m.a[4] + m.a[5] * c);
}

// T_pf(n, L - n) - T_pf(0, L) as a polynomial in n (no cancellation between
// two large prefill times).
__device__ __forceinline__ float recompute_raw(const DevModel& m, float n, float L) {
  return n * (m.k1 + m.k2 * L + m.k3 * n);
}

struct Lat {
  float tpot, ttft;
};

// Eq. 10 (decode term of Eq. 8 for the projected batch and context, scaled
// by the segment's EMA factor; prefill interference amortised over the
// median output length, only on a busy instance) and Eq. 4's TTFT with the
// queue estimate a0 Q + a1 P.
__device__ __forceinline__ Lat latency(const DevModel& m, const InstState& st, float n, float c,
                                       int64_t L) {
  const float tp = t_prefill(m, n, c);
  const float* sg = m.seg[st.seg];
  const float t_iter = sg[3] * (sg[0] + sg[1] * (float)st.A1 + sg[2] * (float)(st.S + L));
  const float interf = st.A1 > 1 ? tp / m.lout1 : 0.0f;
  Lat r;
  r.tpot = t_iter + interf;
  r.ttft = tp + m.a[0] * (float)st.Q + m.a[1] * (float)st.P;
  return r;
}

__device__ __forceinline__ bool eligible(const DevModel& m, int32_t A1, int64_t S, int64_t L) {
  return A1 <= m.b_max && S + L <= m.kv_cap;
}

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

// Bits at positions 0, 8, ..., 56 of x gathered into bits 0..7 (the
// products of the distinct powers of two never collide or carry).
__device__ __forceinline__ uint32_t gather_octet_bits(uint64_t x) {
  return (uint32_t)(((x & 0x0101010101010101ull) * 0x0102040810204080ull) >> 56);
}

__device__ __forceinline__ uint16_t encode_hit(uint32_t h) {
  return (uint16_t)(h > kHitMax ? kHitOverflow : h);
}

__device__ __forceinline__ bool test_bit(const uint64_t* bm, uint32_t i) {
  return ((bm[i >> 6] >> (i & 63)) & 1ull) != 0ull;
}

// Hit of every request on every instance by direct probing: the first block
// on all instances (octets of lanes over instances, 64 per step), then a
// deep walk of each instance that holds it.
__global__ __launch_bounds__(64) void probe_all_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  const int32_t n_inst = a.n_inst;
  for (int32_t r = blockIdx.x; r < a.n_req; r += gridDim.x) {
    const ps_req q = a.reqs[r];
    if (!req_valid(q, a.pool_len)) {
      for (int32_t i = lane; i < n_inst; i += 64) a.hits_out[(size_t)r * n_inst + i] = 0xFFFFFFFFu;
      continue;
    }
    const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
    const int32_t ell = c.len;
    const int32_t nst = ell < kStage ? ell : kStage;
    __syncthreads();
    for (int32_t j = lane; j < nst; j += 64) stage[j] = chain_global(c, j);
    __syncthreads();
    const uint64_t k0 = ell > 0 ? stage[0] : 0ull;
    for (int32_t base = 0; base < n_inst; base += 64) {
      const uint64_t E = __ballot(base + lane < n_inst);
      uint64_t val[kBreadthRounds];
      uint32_t bkt[kBreadthRounds];
#pragma unroll
      for (int rr = 0; rr < kBreadthRounds; ++rr) {
        const int k = rr * 8 + g;
        bkt[rr] = bucket_of(k0, (uint32_t)(base + k), a.t.shift);
        val[rr] = 0ull;
        if (((E >> k) & 1ull) && k0 != 0ull)
          val[rr] = table_of(a.t, (uint32_t)(base + k))[(size_t)bkt[rr] * kSlotsPerBucket + s];
      }
      uint64_t F = 0ull;  // bit k: instance base + k holds the first block
#pragma unroll
      for (int rr = 0; rr < kBreadthRounds; ++rr) {
        const int k = rr * 8 + g;
        const bool act = ((E >> k) & 1ull) != 0ull;
        uint32_t st = octet_status(val[rr], k0, act, g);
        st = octet_resolve(a.t, table_of(a.t, (uint32_t)(base + k)), bkt[rr], k0, st, s, g);
        F |= (uint64_t)gather_octet_bits(__ballot(st == 1u && s == 0)) << (8 * rr);
      }
      uint32_t h = (uint32_t)((F >> lane) & 1ull);
      uint64_t deep = ell > 1 ? F : 0ull;
      while (deep) {
        const int k = __builtin_ctzll(deep);
        deep &= deep - 1;
        const uint32_t hk = deep_walk<true>(a.t, (uint32_t)(base + k), c, stage, 1, g, s);
        if (lane == k) h = hk;
      }
      if (base + lane < n_inst) a.hits_out[(size_t)r * n_inst + base + lane] = h;
    }
  }
}

// Per-lane accumulation over candidates of A: the selector's key over T
// (for H-C-Q a sortable headroom plus the rest of the key), the fallback
// key over C, and |C|, |T|.
struct Acc {
  uint64_t keyT, keyF;
  uint32_t hroom;
  uint32_t nC, nT;
};

// Order-preserving map of a float to u32 (negative values below positive).
__device__ __forceinline__ uint32_t sortable_bits(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t dcq_key(const InstState& st, uint32_t v, uint32_t i) {
  return ((uint64_t)(PS_MAX_DQ - st.D) << 52) | ((uint64_t)(PS_MAX_CHAIN - v) << 28) |
         ((uint64_t)st.Q << 16) | (uint64_t)i;
}

// Packed key of a member of T under selector `sel` (smaller = preferred;
// the id in the low 16 bits ends every order).  H-C-Q: the part after the
// headroom.
__device__ __forceinline__ uint64_t select_key(uint32_t sel, const InstState& st, uint32_t v,
                                               uint32_t i, uint64_t lm) {
  const uint64_t d = (uint64_t)(PS_MAX_DQ - st.D) << 52;
  const uint64_t c = (uint64_t)(PS_MAX_CHAIN - v);
  switch (sel) {
    case PS_SEL_D: return d | i;
    case PS_SEL_DQ: return d | ((uint64_t)st.Q << 16) | i;
    case PS_SEL_DC: return d | (c << 28) | i;
    case PS_SEL_DQC: return d | ((uint64_t)st.Q << 40) | (c << 16) | i;
    case PS_SEL_HCQ: return (c << 28) | ((uint64_t)st.Q << 16) | i;
    case PS_SEL_LMETRIC: return (lm << 16) | i;
    default: return dcq_key(st, v, i);
  }
}

// Membership of candidate (instance i, hit v) of A in C and T, with the
// state and latencies it needs.
struct Member {
  bool inC, inT;
  InstState st;
  Lat lt;
  int64_t n_tok;
};

__device__ __forceinline__ Member member(const ScoreArgs& a, const DevModel& m, uint32_t i,
                                         uint32_t v, int64_t L, float Lf, float wmin, float Z,
                                         bool kvc, float slo) {
  Member r{};
  const int64_t c_tok = (int64_t)v * m.bs;
  r.n_tok = L - c_tok;
  const float n = (float)r.n_tok;
  if (kvc) {
    const float W = fmaxf(0.0f, recompute_raw(m, n, Lf));
    if (!((W - wmin) / Z <= m.eta)) return r;
  }
  r.inC = true;
  r.st = a.inst[i];
  r.lt = latency(m, r.st, n, (float)c_tok, L);
  const bool tpot_ok = (m.flags & PS_F_NO_TPOT_FILTER) || r.lt.tpot < m.tau;
  const bool ttft_ok = !(m.flags & PS_F_TTFT_ADMIT) || r.lt.ttft <= slo;
  r.inT = tpot_ok && ttft_ok;
  return r;
}

__device__ __forceinline__ void evaluate(const ScoreArgs& a, const DevModel& m, Acc& acc,
                                         uint32_t i, uint32_t v, int64_t L, float Lf, float wmin,
                                         float Z, bool kvc, float slo) {
  const Member mb = member(a, m, i, v, L, Lf, wmin, Z, kvc, slo);
  if (!mb.inC) return;
  ++acc.nC;
  const uint64_t lm = (uint64_t)(mb.st.P + mb.n_tok) * (uint64_t)mb.st.A1;
  const uint64_t kf = (m.flags & PS_F_FALLBACK_DCQ) ? dcq_key(mb.st, v, i) : ((lm << 16) | i);
  acc.keyF = kf < acc.keyF ? kf : acc.keyF;
  if (!mb.inT) return;
  ++acc.nT;
  if (m.sel == PS_SEL_RANDOM) return;
  const uint64_t kt = select_key(m.sel, mb.st, v, i, lm);
  if (m.sel == PS_SEL_HCQ) {
    const uint32_t h = sortable_bits(m.tau - mb.lt.tpot);
    if (h < acc.hroom || (h == acc.hroom && kt < acc.keyT)) {
      acc.hroom = h;
      acc.keyT = kt;
    }
  } else {
    acc.keyT = kt < acc.keyT ? kt : acc.keyT;
  }
}

// The (r + 1)-th output of a SplitMix64 stream seeded with `seed`
// (Steele, Lea, Flood; Vigna's public-domain reference).
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, int64_t r) {
  uint64_t z = seed + (uint64_t)(r + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// LDS of one scoring wave: chain stage | live bitmap | next bitmap |
// candidate bitmap (instances holding the first block) | 64 candidate ids |
// u16 hit slots (or device scratch for large pools).
template <bool HITS_IN_LDS>
__global__ __launch_bounds__(64) void score_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int32_t n_inst = a.n_inst;
  const int32_t nw = (n_inst + 63) >> 6;
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem);
  uint64_t* bmA = stage + kStage;
  uint64_t* bmN = bmA + nw;
  uint64_t* bmC = bmN + nw;
  uint16_t* cl = reinterpret_cast<uint16_t*>(bmC + nw);
  uint16_t* hits = HITS_IN_LDS ? cl + 64 : a.scratch + (size_t)blockIdx.x * (size_t)n_inst;
  const int lane = threadIdx.x;
  const int g = lane >> 3, s = lane & 7;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  const DevModel& m = *a.model;

  for (int32_t w = lane; w < 3 * nw; w += 64) bmA[w] = 0ull;

  for (int32_t r = blockIdx.x; r < a.n_req; r += gridDim.x) {
    const ps_req q = a.reqs[r];
    if (!req_valid(q, a.pool_len)) {
      if (lane == 0) {
        a.out[r] = ps_result{-1, 0, 0.0f, 0.0f, PS_R_INVALID};
        if (a.sizes) a.sizes[3 * (size_t)r] = a.sizes[3 * (size_t)r + 1] = a.sizes[3 * (size_t)r + 2] = 0;
      }
      continue;
    }
    const ChainRef c{a.pool + q.pre_off, a.pool + q.tail_off, q.pre_len, q.pre_len + q.tail_len};
    const int32_t ell = c.len;
    const int64_t L = (int64_t)ell * m.bs;
    const float Lf = (float)L;
    const int32_t nst = ell < kStage ? ell : kStage;
    __syncthreads();
    for (int32_t j = lane; j < nst; j += 64) stage[j] = chain_global(c, j);
    __syncthreads();

    // |A|: capacity-eligible instances are those with room >= L.
    const uint32_t nA = (uint32_t)(n_inst - wave_lower_bound(a.room_sorted, n_inst, L, lane));

    // (1) Holders of the first block among the eligible instances.
    uint32_t nCand = 0;
    if (nA > 0 && ell > 0) {
      const IdxHit h0 = index_lookup(a.x, stage[0], g == 0, g, s);
      const bool found0 = __shfl(h0.found ? 1 : 0, 0) != 0;
      const uint32_t off0 = __shfl(h0.off, 0), cnt0 = __shfl(h0.cnt, 0);
      if (found0 && cnt0 > kPopular) {  // holders as a bitmap: lanes over its words
        const uint64_t* bm = a.x.bitmaps + (size_t)off0 * a.x.nw;
        for (int32_t w0 = 0; w0 < nw; w0 += 64) {
          const int32_t w = w0 + lane;
          uint64_t d = w < nw ? bm[w] : 0ull, el_bits = 0ull;
          while (d) {
            const int b = __builtin_ctzll(d);
            d &= d - 1;
            if (a.room[w * 64 + b] >= L) el_bits |= 1ull << b;
          }
          const uint32_t cntl = (uint32_t)__popcll(el_bits);
          uint32_t rank = nCand + wave_exclusive_sum(cntl, lane);
          if (w < nw) bmC[w] = el_bits;
          uint64_t e2 = el_bits;
          while (e2 && rank < 64) {
            const int b = __builtin_ctzll(e2);
            e2 &= e2 - 1;
            cl[rank++] = (uint16_t)(w * 64 + b);
          }
          nCand += wave_sum_u32(cntl);
        }
      } else if (found0) {
        for (uint32_t t0 = 0; t0 < cnt0; t0 += 64) {
          const uint32_t t = t0 + lane;
          const uint32_t id = t < cnt0 ? a.x.holders[off0 + t] : 0u;
          const bool el = t < cnt0 && a.room[id] >= L;
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
    if (few) {
      if ((uint32_t)lane < nCand) myid = cl[lane];
      for (uint32_t k = 0; k < nCand; ++k) {
        const uint32_t id = (uint32_t)__shfl((int)myid, (int)k);
        const uint32_t hk = ell > 1 ? run_walk<true>(a.t, id, c, stage, 0, g, s) : 1u;
        if ((uint32_t)lane == k) myhit = hk;
      }
      if ((uint32_t)lane < nCand) hits[myid] = encode_hit(myhit);
    } else {
      for (int32_t w = lane; w < nw; w += 64) bmA[w] = bmC[w];
      __syncthreads();
      uint32_t nalive = nCand;
      int32_t p = 1;
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
          const uint32_t hk = run_walk<true>(a.t, who, c, stage, p, g, s);
          if (lane == 0) {
            hits[who] = encode_hit(hk);
            bmA[who >> 6] = 0ull;
          }
          nalive = 0;
          __syncthreads();
          break;
        }
        const int32_t jq = p + g;
        const uint64_t kq = jq < ell ? ((jq < kStage) ? stage[jq] : chain_global(c, jq)) : 0ull;
        const IdxHit hq = index_lookup(a.x, kq, jq < ell, g, s);
        int32_t used = 0;
        for (int t = 0; t < 8; ++t) {
          const int32_t pos = p + t;
          if (pos >= ell || nalive <= 1) break;
          const bool f = __shfl(hq.found ? 1 : 0, 8 * t) != 0;
          const uint32_t off = __shfl(hq.off, 8 * t), cnt = __shfl(hq.cnt, 8 * t);
          if (f && cnt > kPopular) {  // live &= holder bitmap, lane-owned words
            const uint64_t* bm = a.x.bitmaps + (size_t)off * a.x.nw;
            uint32_t live = 0;
            for (int32_t w = lane; w < nw; w += 64) {
              const uint64_t aw = bmA[w];
              const uint64_t nwd = aw & bm[w];
              uint64_t d = aw & ~nwd;
              while (d) {
                const int b = __builtin_ctzll(d);
                d &= d - 1;
                hits[w * 64 + b] = encode_hit((uint32_t)pos);
              }
              bmA[w] = nwd;
              live += (uint32_t)__popcll(nwd);
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
          for (int32_t w = lane; w < nw; w += 64) {
            const uint64_t aw = bmA[w], nwd = bmN[w];
            uint64_t d = aw & ~nwd;
            while (d) {
              const int b = __builtin_ctzll(d);
              d &= d - 1;
              hits[w * 64 + b] = encode_hit((uint32_t)pos);
            }
            bmA[w] = nwd;
            bmN[w] = 0ull;
            live += (uint32_t)__popcll(nwd);
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
            hits[w * 64 + b] = encode_hit((uint32_t)ell);
          }
          bmA[w] = 0ull;
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
          const uint32_t hk = run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
          if (lane == k) v = hk;
        }
        if (cand) {
          const float W = fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)v * m.bs), Lf));
          const uint32_t wb = __float_as_uint(W);
          wmin_bits = wb < wmin_bits ? wb : wmin_bits;
        }
      }
    }
    const float wmin = __uint_as_float((uint32_t)wave_min_u64((uint64_t)wmin_bits));

    // (3)-(4) Filters and keys.  The hit-0 class is visited only if its
    // common penalty passes Eq. 9.
    const float tpf_cold = t_prefill(m, Lf, 0.0f);
    const float slo = fmaxf(m.ttft_floor, tpf_cold);
    const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;
    const bool admit0 = n0 > 0 && (!kvc || (W0 - wmin) / Z <= m.eta);
    Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
    if (nA > 0) {
      if (few) {
        if ((uint32_t)lane < nCand) evaluate(a, m, acc, myid, myhit, L, Lf, wmin, Z, kvc, slo);
      } else {
        for (int32_t base = 0; base < n_inst; base += 64) {
          const int32_t i = base + lane;
          const bool cand = i < n_inst && test_bit(bmC, (uint32_t)i);
          uint32_t v = cand ? hits[i] : 0u;
          uint64_t ovf = __ballot(cand && v == kHitOverflow);
          while (ovf) {
            const int k = __builtin_ctzll(ovf);
            ovf &= ovf - 1;
            const uint32_t hk = run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
            if (lane == k) v = hk;
          }
          if (cand) evaluate(a, m, acc, (uint32_t)i, v, L, Lf, wmin, Z, kvc, slo);
        }
      }
      if (admit0) {
        // The eligible non-holders (hit 0) share n = L.  Without set sizes
        // to report, only the best packing key of that class matters: the
        // first member of T in key order (decoding desc, queued asc, id
        // asc).  The whole class is evaluated when sizes are requested or
        // when no member is in T (then the fallback key may come from it).
        bool done0 = false;
        const bool keyed = m.sel == PS_SEL_DCQ || m.sel == PS_SEL_DQ || m.sel == PS_SEL_DQC;
        if (!a.sizes && keyed) {
          for (int32_t base = 0; base < n_inst && !done0; base += 64) {
            const int32_t k = base + lane;
            bool ok = false;
            uint32_t i = 0;
            if (k < n_inst) {
              i = a.order0[k];
              if (a.room[i] >= L && !test_bit(bmC, i)) {
                const InstState st = a.inst[i];
                const Lat lt = latency(m, st, Lf, 0.0f, L);
                ok = ((m.flags & PS_F_NO_TPOT_FILTER) || lt.tpot < m.tau) &&
                     (!(m.flags & PS_F_TTFT_ADMIT) || lt.ttft <= slo);
              }
            }
            const uint64_t okm = __ballot(ok);
            if (okm) {
              if (lane == __builtin_ctzll(okm)) {
                const InstState st = a.inst[i];
                const uint64_t kt = select_key(m.sel, st, 0u, i, 0ull);
                acc.keyT = kt < acc.keyT ? kt : acc.keyT;
              }
              done0 = true;
            }
          }
        }
        if (!done0) {
          for (int32_t base = 0; base < n_inst; base += 64) {
            const int32_t i = base + lane;
            if (i < n_inst && !test_bit(bmC, (uint32_t)i) && a.room[i] >= L)
              evaluate(a, m, acc, (uint32_t)i, 0u, L, Lf, wmin, Z, kvc, slo);
          }
        }
      }
    }
    uint64_t keyT;
    if (m.sel == PS_SEL_HCQ) {  // smallest headroom first, then the rest of the key
      const uint64_t hmin = wave_min_u64((uint64_t)acc.hroom);
      keyT = wave_min_u64((uint64_t)acc.hroom == hmin ? acc.keyT : ~0ull);
    } else {
      keyT = wave_min_u64(acc.keyT);
    }
    const uint64_t keyF = wave_min_u64(acc.keyF);
    const uint32_t nC = wave_sum_u32(acc.nC);
    const uint32_t nT = wave_sum_u32(acc.nT);
    if (m.sel == PS_SEL_RANDOM && nT > 0) {
      // the k-th member of T in id order
      const uint64_t z = splitmix64_at(m.rand_seed, r);
      const uint32_t kth = (uint32_t)(((z >> 32) * (uint64_t)nT) >> 32);
      uint32_t seen = 0;
      for (int32_t base = 0; base < n_inst; base += 64) {
        const int32_t i = base + lane;
        const bool el = i < n_inst && a.room[i] >= L;
        const bool cand = el && test_bit(bmC, (uint32_t)i);
        uint32_t v = cand ? hits[i] : 0u;
        uint64_t ovf = __ballot(cand && v == kHitOverflow);
        while (ovf) {
          const int k = __builtin_ctzll(ovf);
          ovf &= ovf - 1;
          const uint32_t hk = run_walk<true>(a.t, (uint32_t)(base + k), c, stage, 0, g, s);
          if (lane == k) v = hk;
        }
        bool inT = false;
        if (el && (cand || admit0)) inT = member(a, m, (uint32_t)i, v, L, Lf, wmin, Z, kvc, slo).inT;
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
          if (v == kHitOverflow) v = run_walk<true>(a.t, best, c, stage, 0, g, s);
        }
      }
      const int64_t c_tok = (int64_t)v * m.bs;
      const InstState st = a.inst[best];
      const Lat lt = latency(m, st, (float)(L - c_tok), (float)c_tok, L);
      if (lt.ttft > slo) fl |= PS_R_TTFT_MISS;
      res = ps_result{(int32_t)best, (int32_t)v, lt.ttft, lt.tpot, fl};
    }
    if (lane == 0) {
      a.out[r] = res;
      if (a.sizes) {
        a.sizes[3 * (size_t)r] = nA;
        a.sizes[3 * (size_t)r + 1] = nC;
        a.sizes[3 * (size_t)r + 2] = nT;
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

__device__ __forceinline__ int32_t segment_of(const DevModel& m, int32_t B) {
  for (int32_t s = 0; s < m.n_seg; ++s)
    if (B <= m.seg_ub[s]) return s;
  return m.n_seg - 1;
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
      __threadfence();  // later probes of this wave must see these inserts
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

// ----------------------------------------------------- per-arrival scheduler
// One wave's share of a workgroup-wide reduction.
struct SeqPart {
  uint64_t keyT, keyF;
  uint32_t hroom, nC, nT, wmin, nA, pad;
};

// Workgroup LDS of the scheduler (a fixed layout, plus the dirty bitmap).
struct SeqShared {
  uint64_t stage[kSeqStage];          // the request's chain head
  SeqPart part[2][kSeqWaves];         // reduction partials (alternating)
  uint32_t cnt[kSeqU][kSeqWaves];     // per-wave counts of one insert step
  uint32_t ext[kExtMax][2];           // hit extensions: instance, first unknown position
  uint32_t ring[3];                   // first-absent minima of the sweeps
  uint32_t n_ext, hit, pick, count;
  int64_t rp;                         // row position found by a run walk's probe
};

__device__ __forceinline__ uint64_t seq_key(const SeqShared& sh, const ChainRef& c, int32_t j) {
  return j < kSeqStage ? sh.stage[j] : chain_global(c, j);
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

    // (1) capacity guard
    uint32_t nA = 0;
    if (!replay && L <= room_ub) {
      uint32_t al = 0;
      uint64_t rl = ~0ull;  // ~(room + 1), minimised (room >= -1)
      for (int32_t i = tid; i < n_inst; i += NT) {
        const InstState st = a.inst[i];
        al += eligible(m, st.A1, st.S, L) ? 1u : 0u;
        const int64_t room = st.A1 <= m.b_max ? m.kv_cap - st.S : -1;
        const uint64_t x = ~((uint64_t)room + 1ull);
        rl = x < rl ? x : rl;
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
    int32_t best = -1;
    uint32_t fl = PS_R_REJECT, nC = 0, nT = 0;
    const float Z = recompute_raw(m, Lf, Lf);  // T_pf(L, 0) - T_pf(0, L)
    const float tpf_cold = t_prefill(m, Lf, 0.0f);
    const float slo = fmaxf(m.ttft_floor, tpf_cold);
    if (work) {
      // (2) live hits
      const int32_t nst = ell < kSeqStage ? ell : kSeqStage;
      for (int32_t j0 = 0; j0 < nst; j0 += 8 * NT) {  // eight loads in flight per thread
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
      if (tid == 0) sh.n_ext = 0u;
      __syncthreads();
      for (int32_t i = tid; i < n_inst; i += NT) {
        if (!test_bit(dirty, (uint32_t)i)) continue;
        if (replay ? i != forced : !eligible(m, a.inst[i].A1, a.inst[i].S, L)) continue;
        const uint32_t v = H[i];
        if ((int32_t)v >= ell) continue;
        if (!probe(a.t, (uint32_t)i, seq_key(sh, c, (int32_t)v))) continue;
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
        for (int32_t i = tid; i < n_inst; i += NT) {
          const InstState st = a.inst[i];
          if (!eligible(m, st.A1, st.S, L)) continue;
          const float W = fmaxf(0.0f, recompute_raw(m, (float)(L - (int64_t)H[i] * m.bs), Lf));
          const uint32_t wb = __float_as_uint(W);
          wl = wb < wl ? wb : wl;
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
        const bool kvc = !(m.flags & PS_F_NO_KVC_FILTER) && Z > 0.0f;

        // (3b) filters and keys
        Acc acc{~0ull, ~0ull, ~0u, 0u, 0u};
        for (int32_t i = tid; i < n_inst; i += NT) {
          const InstState st = a.inst[i];
          if (eligible(m, st.A1, st.S, L))
            evaluate(sa, m, acc, (uint32_t)i, H[i], L, Lf, wmin, Z, kvc, slo);
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

    // (4) result and commit
    if (best >= 0 && best % NT == tid) {
      const uint32_t v = H[best];
      const int64_t c_tok = (int64_t)v * m.bs;
      InstState st = a.inst[best];
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
}

}  // namespace

// ------------------------------------------------------------------ launchers
size_t ps_score_lds_bytes(int32_t n_inst) {
  const size_t nw = ((size_t)n_inst + 63) / 64;
  const size_t hits = ps_hits_fit_lds(n_inst) ? (size_t)n_inst * sizeof(uint16_t) : 0;
  return (size_t)kStage * sizeof(uint64_t) + 3 * nw * sizeof(uint64_t) + 64 * sizeof(uint16_t) +
         (hits + 15) / 16 * 16;
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

hipError_t ps_launch_score(const ScoreArgs& a, bool hits_in_lds, int grid, bool probe_all,
                           hipStream_t s) {
  if (a.n_req == 0) return hipSuccess;
  if (probe_all) {
    hipLaunchKernelGGL(probe_all_kernel, dim3(grid), dim3(64), (size_t)kStage * sizeof(uint64_t), s,
                       a);
  } else {
    const size_t lds = ps_score_lds_bytes(a.n_inst);
    if (hits_in_lds)
      hipLaunchKernelGGL(score_kernel<true>, dim3(grid), dim3(64), lds, s, a);
    else
      hipLaunchKernelGGL(score_kernel<false>, dim3(grid), dim3(64), lds, s, a);
  }
  return hipGetLastError();
}

hipError_t ps_launch_commit(const CommitArgs& a, hipStream_t s) {
  if (a.n_grp == 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3(a.n_grp), dim3(64), 0, s, a);
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
