// Device helpers shared by the kernels of the window scorer and of the
// per-arrival scheduler (gfx950, wave64): DPP wave reductions, bucket probes
// and compare-and-swap inserts of the per-instance tables, prefix walks, the
// latency model, and the evaluation of one candidate (membership in C and T
// and its packing keys).  Internal to this library.
#pragma once

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

template <int CTRL, int RM>
__device__ __forceinline__ void min32_step(uint32_t& v) {
  const uint32_t t = dpp_src<CTRL, RM>(0xFFFFFFFFu, v);
  v = t < v ? t : v;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  min32_step<0x111, 0xF>(v);
  min32_step<0x112, 0xF>(v);
  min32_step<0x114, 0xF>(v);
  min32_step<0x118, 0xF>(v);
  min32_step<0x142, 0xA>(v);
  min32_step<0x143, 0xC>(v);
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
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

// A 64-bit value of lane src (a wave-uniform result).
__device__ __forceinline__ int64_t lane_value64(int64_t v, int src) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, src);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), src);
  return (int64_t)(((uint64_t)hi << 32) | lo);
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
// the bucket reads of DR x 8 positions (DR loads per lane in flight), then
// prefetches the next step's chain hashes, then evaluates in chain order
// and stops at the first absent position.  Positions below kStage read the LDS copy of the chain.
// Wave-uniform arguments; returns the hit.
template <bool STAGED, int DR = kDeepRounds>
__device__ uint32_t deep_walk(const Tables& t, uint32_t inst, const ChainRef& c,
                              const uint64_t* stage, int32_t pos, int g, int s) {
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, inst);
  uint64_t nk[DR];
#pragma unroll
  for (int r = 0; r < DR; ++r) {
    const int32_t j = pos + r * 8 + g;
    nk[r] = 0ull;
    if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
  }
  while (pos < ell) {
    uint64_t key[DR], val[DR];
    uint32_t b[DR];
#pragma unroll
    for (int r = 0; r < DR; ++r) {
      const int32_t j = pos + r * 8 + g;
      key[r] = nk[r];
      b[r] = bucket_of(key[r], inst, t.shift);
      val[r] = 0ull;
      if (j < ell && key[r] != 0ull) val[r] = tab[(size_t)b[r] * kSlotsPerBucket + s];
    }
    const int32_t next = pos + DR * 8;
#pragma unroll
    for (int r = 0; r < DR; ++r) {
      const int32_t j = next + r * 8 + g;
      nk[r] = 0ull;
      if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
    }
#pragma unroll
    for (int r = 0; r < DR; ++r) {
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

// Lane probing: one lane reads the whole 64-byte bucket of its own key
// (four 16-byte loads).  1 found, 0 absent (an empty slot ends the probe
// sequence, and the zero hash is never stored), 2 full bucket without the
// key (the next bucket decides).
__device__ __forceinline__ uint32_t lane_status(const Bucket& bk, uint64_t key) {
  bool f = false, e = false;
#pragma unroll
  for (int s = 0; s < kSlotsPerBucket; ++s) {
    f |= bk.k[s] == key;
    e |= bk.k[s] == 0ull;
  }
  if (key == 0ull) return 0u;
  return f ? 1u : (e ? 0u : 2u);
}

// Linear probing past full buckets for one lane (rare at load factor <= 0.5);
// true when the key is found.
__device__ __noinline__ bool lane_resolve(const Tables& t, const uint64_t* tab, uint32_t b,
                                          uint64_t key) {
  for (uint32_t step = 1; step <= t.bmask; ++step) {
    b = (b + 1) & t.bmask;
    const uint32_t st = lane_status(load_bucket(tab + (size_t)b * kSlotsPerBucket), key);
    if (st != 2u) return st == 1u;
  }
  return false;
}

// Deep walk with lane probing: positions pos.. of the chain on one
// instance, DR x 64 per step (lane l takes pos + 64 r + l), the next step's
// keys read while the buckets are in flight.  Wave-uniform arguments;
// returns the first position whose block the instance does not hold.
template <bool STAGED, int DR>
__device__ uint32_t lane_walk(const Tables& t, uint32_t inst, const ChainRef& c,
                              const uint64_t* stage, int32_t pos, int lane) {
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, inst);
  uint64_t nk[DR];
#pragma unroll
  for (int r = 0; r < DR; ++r) {
    const int32_t j = pos + r * 64 + lane;
    nk[r] = 0ull;
    if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
  }
  while (pos < ell) {
    uint64_t key[DR];
    uint32_t b[DR];
    Bucket v[DR];
#pragma unroll
    for (int r = 0; r < DR; ++r) {
      const int32_t j = pos + r * 64 + lane;
      key[r] = nk[r];
      b[r] = bucket_of(key[r], inst, t.shift);
      v[r] = Bucket{};
      if (j < ell && key[r] != 0ull) v[r] = load_bucket(tab + (size_t)b[r] * kSlotsPerBucket);
    }
    const int32_t next = pos + DR * 64;
#pragma unroll
    for (int r = 0; r < DR; ++r) {
      const int32_t j = next + r * 64 + lane;
      nk[r] = 0ull;
      if (j < ell) nk[r] = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
    }
#pragma unroll
    for (int r = 0; r < DR; ++r) {
      const int32_t j = pos + r * 64 + lane;
      const bool act = j < ell;
      uint32_t st = act ? lane_status(v[r], key[r]) : 1u;
      if (st == 2u) st = lane_resolve(t, tab, b[r], key[r]) ? 1u : 0u;
      const uint64_t miss = __ballot(st != 1u);
      if (miss) return (uint32_t)(pos + r * 64 + __builtin_ctzll(miss));
    }
    pos = next;
  }
  return (uint32_t)ell;
}

// One compare step of a row walk: chain positions q.. against row entries
// k.., U x 64 of them (U per lane, coalesced).  Returns the first position
// whose block differs from the row entry (or lies past the row's end), or
// -1 when all of them match.
template <bool STAGED, int U>
__device__ __forceinline__ int32_t run_compare(const ChainRef& c, const uint64_t* stage,
                                               const uint64_t* row, int64_t rlen, int32_t q,
                                               int64_t k, int lane) {
  const int32_t ell = c.len;
  bool mism[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int32_t j = q + 64 * u + lane;
    const int64_t kk = k + 64 * u + lane;
    const bool valid = j < ell;
    uint64_t cj = 0ull, rk = 0ull;
    if (valid) cj = (STAGED && j < kStage) ? stage[j] : chain_global(c, j);
    if (valid && kk < rlen) rk = row[kk];
    mism[u] = valid && (kk >= rlen || cj != rk);
  }
  int32_t next = -1;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint64_t mm = __ballot(mism[u]);
    if (next < 0 && mm) next = q + 64 * u + __builtin_ctzll(mm);
  }
  return next;
}

// Walk of one instance along its row: one octet probe finds the block at
// `pos` and its row position; the chain blocks after it are compared with
// the row entries after it, 256 per step (4 per lane, coalesced; W per lane
// after the first step), and the first mismatch is probed again (it may
// begin another run of the row, e.g. after a shared system prompt).  A run
// shorter than 8 blocks hands the rest of the walk to the octet walk.
// Wave-uniform arguments; returns the hit.  U0 = positions per lane in the
// first step; key_at: the chain's block at `pos` when the caller has it (0:
// read it).
template <bool STAGED, int W = kWalkU, int U0 = 4>
__device__ __forceinline__ uint32_t run_walk(const Tables& t, uint32_t inst, const ChainRef& c,
                             const uint64_t* stage, int32_t pos, int g, int s,
                             uint64_t key_at = 0ull) {
  const int lane = g * 8 + s;
  const int32_t ell = c.len;
  const uint64_t* tab = table_of(t, inst);
  const uint64_t* row = t.rows + (size_t)inst * (size_t)t.row_cap;
  const int64_t rlen = t.count[inst];
  while (pos < ell) {
    const uint64_t key = key_at != 0ull ? key_at
                         : (STAGED && pos < kStage) ? stage[pos] : chain_global(c, pos);
    key_at = 0ull;
    if (key == 0ull) return (uint32_t)pos;
    uint32_t b = bucket_of(key, inst, t.shift);
    int64_t rp = -1;
    bool decided = false;
    for (uint32_t step = 0; step <= t.bmask && !decided; ++step) {
      // each slot's row position is read with the slot (no second trip)
      const uint64_t val = g == 0 ? tab[(size_t)b * kSlotsPerBucket + s] : 0ull;
      const uint32_t rpv =
          g == 0 ? t.rowpos[(size_t)inst * t.slots + (size_t)b * kSlotsPerBucket + s] : 0u;
      const uint64_t fm = __ballot(g == 0 && val == key) & 0xFFull;
      const uint64_t em = __ballot(g == 0 && val == 0ull) & 0xFFull;
      if (fm) {
        rp = (uint32_t)__shfl((int)rpv, __builtin_ctzll(fm));
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
    // The first step compares U0 positions per lane; a run that goes on is
    // likely long (a session prefix), so later steps compare W per lane.
    int32_t next = run_compare<STAGED, U0>(c, stage, row, rlen, q, k, lane);
    q += 64 * U0;
    k += 64 * U0;
    while (next < 0) {
      if (q >= ell) return (uint32_t)ell;
      next = run_compare<STAGED, W>(c, stage, row, rlen, q, k, lane);
      q += 64 * W;
      k += 64 * W;
    }
    if (next - start < 8) return deep_walk<STAGED>(t, inst, c, stage, next, g, s);
    pos = next;
  }
  return (uint32_t)ell;
}

// The model in LDS for the launch of a persistent kernel.  Read through the
// device pointer, every field is a global load that the compiler repeats,
// and waits for, after each store of the kernel's loop (the pointer may
// alias them); the LDS copy is read with LDS loads.  Every lane of the
// workgroup calls it; the copy is visible after the next barrier.
__device__ __forceinline__ void stage_model(DevModel& dst, const DevModel* src, int tid,
                                            int nthreads) {
  static_assert(sizeof(DevModel) % 4 == 0, "the model is copied in 4-byte words");
  for (int k = tid; k < (int)(sizeof(DevModel) / 4); k += nthreads)
    reinterpret_cast<uint32_t*>(&dst)[k] = reinterpret_cast<const uint32_t*>(src)[k];
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
// Eq. 8's decode-iteration time with the request's L tokens added to S.
__device__ __forceinline__ float t_iter_of(const DevModel& m, const InstState& st, int64_t L) {
  const float* sg = m.seg[st.seg];
  return sg[3] * (sg[0] + sg[1] * (float)st.A1 + sg[2] * (float)(st.S + L));
}

__device__ __forceinline__ Lat latency(const DevModel& m, const InstState& st, float n, float c,
                                       int64_t L) {
  const float tp = t_prefill(m, n, c);
  const float t_iter = t_iter_of(m, st, L);
  const float interf = st.A1 > 1 ? tp / m.lout1 : 0.0f;
  Lat r;
  r.tpot = t_iter + interf;
  r.ttft = tp + m.a[0] * (float)st.Q + m.a[1] * (float)st.P;
  return r;
}

// Another lane's state (every lane must call it).
__device__ __forceinline__ InstState shfl_state(const InstState& st, int src) {
  InstState r;
  r.D = __shfl(st.D, src);
  r.Q = __shfl(st.Q, src);
  r.A1 = __shfl(st.A1, src);
  r.seg = __shfl(st.seg, src);
  r.P = __shfl(st.P, src);
  r.S = __shfl(st.S, src);
  return r;
}

__device__ __forceinline__ bool eligible(const DevModel& m, int32_t A1, int64_t S, int64_t L) {
  return A1 <= m.b_max && S + L <= m.kv_cap;
}

// Bits at positions 0, 8, ..., 56 of x gathered into bits 0..7 (the
// products of the distinct powers of two never collide or carry).
__device__ __forceinline__ uint32_t gather_octet_bits(uint64_t x) {
  return (uint32_t)(((x & 0x0101010101010101ull) * 0x0102040810204080ull) >> 56);
}

__device__ __forceinline__ uint16_t encode_hit(uint32_t h) {
  return (uint16_t)(h > kHitMax ? kHitOverflow : h);
}

// bit i of a bitmap of 64-bit words, read as its 32-bit half (a 32-bit
// shift instead of a 64-bit one: the scorers are bound by VALU issue)
__device__ __forceinline__ bool test_bit(const uint64_t* bm, uint32_t i) {
  return ((reinterpret_cast<const uint32_t*>(bm)[i >> 5] >> (i & 31u)) & 1u) != 0u;
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

// `state()` supplies the instance's load state; it is called only for
// members of C.
// KEYED: the caller guarantees a keyed selector (D-C-Q, D-Q, D-Q-C) and no
// TTFT admission, so those branches compile away.
template <bool KEYED = false, class State>
__device__ __forceinline__ Member member_with(const DevModel& m, State state, uint32_t v,
                                              int64_t L, float Lf, float wmin, float Z, bool kvc,
                                              float slo) {
  Member r{};
  const int64_t c_tok = (int64_t)v * m.bs;
  r.n_tok = L - c_tok;
  const float n = (float)r.n_tok;
  if (kvc) {
    const float W = fmaxf(0.0f, recompute_raw(m, n, Lf));
    if (!((W - wmin) / Z <= m.eta)) return r;
  }
  r.inC = true;
  r.st = state();
  r.lt = latency(m, r.st, n, (float)c_tok, L);
  const bool tpot_ok = (m.flags & PS_F_NO_TPOT_FILTER) || r.lt.tpot < m.tau;
  const bool ttft_ok = KEYED || !(m.flags & PS_F_TTFT_ADMIT) || r.lt.ttft <= slo;
  r.inT = tpot_ok && ttft_ok;
  return r;
}

__device__ __forceinline__ Member member(const ScoreArgs& a, const DevModel& m, uint32_t i,
                                         uint32_t v, int64_t L, float Lf, float wmin, float Z,
                                         bool kvc, float slo) {
  return member_with(m, [&]() { return a.inst[i]; }, v, L, Lf, wmin, Z, kvc, slo);
}

template <bool KEYED = false, class State>
__device__ __forceinline__ void evaluate_with(const DevModel& m, Acc& acc, uint32_t i, uint32_t v,
                                              State state, int64_t L, float Lf, float wmin,
                                              float Z, bool kvc, float slo) {
  const Member mb = member_with<KEYED>(m, state, v, L, Lf, wmin, Z, kvc, slo);
  if (!mb.inC) return;
  ++acc.nC;
  const uint64_t lm = (uint64_t)(mb.st.P + mb.n_tok) * (uint64_t)mb.st.A1;
  const uint64_t kf = (m.flags & PS_F_FALLBACK_DCQ) ? dcq_key(mb.st, v, i) : ((lm << 16) | i);
  acc.keyF = kf < acc.keyF ? kf : acc.keyF;
  if (!mb.inT) return;
  ++acc.nT;
  if (!KEYED && m.sel == PS_SEL_RANDOM) return;
  const uint64_t kt = select_key(m.sel, mb.st, v, i, lm);
  if (!KEYED && m.sel == PS_SEL_HCQ) {
    const uint32_t h = sortable_bits(m.tau - mb.lt.tpot);
    if (h < acc.hroom || (h == acc.hroom && kt < acc.keyT)) {
      acc.hroom = h;
      acc.keyT = kt;
    }
  } else {
    acc.keyT = kt < acc.keyT ? kt : acc.keyT;
  }
}

__device__ __forceinline__ void evaluate(const ScoreArgs& a, const DevModel& m, Acc& acc,
                                         uint32_t i, uint32_t v, int64_t L, float Lf, float wmin,
                                         float Z, bool kvc, float slo) {
  evaluate_with(m, acc, i, v, [&]() { return a.inst[i]; }, L, Lf, wmin, Z, kvc, slo);
}

// The (r + 1)-th output of a SplitMix64 stream seeded with `seed`
// (Steele, Lea, Flood; Vigna's public-domain reference).
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, int64_t r) {
  uint64_t z = seed + (uint64_t)(r + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ int32_t segment_of(const DevModel& m, int32_t B) {
  for (int32_t s = 0; s < m.n_seg; ++s)
    if (B <= m.seg_ub[s]) return s;
  return m.n_seg - 1;
}

}  // namespace
