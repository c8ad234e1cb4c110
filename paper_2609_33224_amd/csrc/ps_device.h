// Internal device-side layout and inline helpers of the window scorer
// (gfx950, wave64).  Shared by the kernels and the host API of this library
// only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "packserve.h"

namespace ps {

constexpr int kStage = 256;            // chain blocks staged in LDS per request (2 KiB)
constexpr int kSlotsPerBucket = 8;     // 8 x 64-bit keys = one 64-byte bucket
constexpr int kDeepRounds = 2;         // octet loads per lane in flight: 16 positions per step
constexpr int kWalkU = 4;             // row-walk positions per lane after the first step
// Per-candidate hit slots (u16 in LDS): exact hits up to kHitMax, then two
// markers.
constexpr uint32_t kHitMax = 0xFFFDu;
constexpr uint32_t kHitOverflow = 0xFFFEu;  // hit > kHitMax: recomputed where needed
constexpr uint32_t kInelig = 0xFFFFu;       // not capacity-eligible
// Per-wave dynamic LDS above which hit slots move to device scratch.
constexpr size_t kLdsHitBudget = 16 * 1024;

// Per-instance load state, 32 bytes (one pair of 16-byte loads).
struct alignas(16) InstState {
  int32_t D;    // decoding
  int32_t Q;    // queued
  int32_t A1;   // D + Q + 1: projected decode batch after admission
  int32_t seg;  // decode segment of A1
  int64_t P;    // pending uncached prefill tokens
  int64_t S;    // context tokens of the active requests
};

// Device copy of the model, with the recomputation-penalty polynomial
// precomputed: T_pf(n, L - n) - T_pf(0, L) = n (k1 + k2 L + k3 n).
struct DevModel {
  float a[6];
  float k1, k2, k3;
  float eta, tau, ttft_floor, lout1;  // lout1 = max(1, lout)
  int32_t bs, b_max;
  int64_t kv_cap;
  uint32_t flags;     // PS_F_* admission bits
  uint32_t sel;       // PS_SEL_*
  uint64_t rand_seed;
  int32_t n_seg;
  // 1 when the zero-hit TPOT test can only turn from pass to fail as L
  // grows (finite coefficients, alpha1, alpha3, every beta2 and gamma >= 0):
  // then an instance's zero-hit admission is one threshold on L.
  uint32_t mono;
  int32_t seg_ub[PS_MAX_SEG];
  float seg[PS_MAX_SEG][4];  // beta0, beta1, beta2, gamma
};

// Table geometry: n_inst tables of (1 << log2_buckets) buckets each.
// Per-instance tables.  Besides the hash slots, every instance keeps its
// distinct cached blocks as a row in insertion order (row_cap entries each;
// row_len = count), and rowpos[slot] gives the row position of the key in
// that slot, so a walk that finds one block can compare the blocks after it
// with the row sequentially.
struct Tables {
  uint64_t* keys;       // n_inst * slots
  uint32_t* count;      // distinct keys per instance (= row length)
  uint32_t* rowpos;     // n_inst * slots: row position of each occupied slot
  uint64_t* rows;       // n_inst * row_cap, insertion order
  int64_t slots;        // slots per instance = buckets * 8
  int64_t row_cap;      // = table cap
  uint32_t bmask;       // buckets - 1
  uint32_t shift;       // 64 - log2(buckets) (64 when one bucket)
};

// Per-instance salted bucket index: a multiply-shift (Fibonacci) hash of the
// key xor an instance salt, so one hash lands at unrelated offsets in
// different tables (no two instances' probes for a request share a channel
// pattern).
__host__ __device__ __forceinline__ uint32_t bucket_of(uint64_t key, uint32_t inst,
                                                       uint32_t shift) {
  uint64_t x = (key ^ (0x9E3779B97F4A7C15ull * (uint64_t)(inst + 1u))) * 0xD6E8FEB86659FD93ull;
  return shift >= 64 ? 0u : (uint32_t)(x >> shift);
}

// Prefix index: every cached block hash of the pool with the ascending list
// of instances holding it (the GPU form of a prefix tree over chained hashes:
// one hash names one prefix).  16-byte entries, buckets of 8 = one 128-byte
// line, multiply-shift bucket with the salt kIndexSalt, linear probing.
// A hash held by more than kPopular instances keeps its holders as a bitmap
// of the pool (nw 64-bit words; `off` = bitmap number); otherwise as an
// ascending list of ids (`off` = first list entry).
struct alignas(16) IdxEntry {
  uint64_t key;   // 0 = empty
  uint32_t off;   // list offset, or bitmap number when cnt > kPopular
  uint32_t cnt;   // number of holders
};
constexpr uint32_t kIndexSalt = 0x10000u;  // not an instance id
constexpr uint32_t kPopular = 64;

struct GIndex {
  IdxEntry* ent;
  uint16_t* holders;
  uint64_t* bitmaps;  // n_popular * nw words
  uint32_t nw;        // words per bitmap = ceil(n_inst / 64)
  uint32_t bmask;
  uint32_t shift;
  uint32_t n_pop;     // bitmaps (hashes with more than kPopular holders)
};

// Prefix groups of one window.  Requests whose chains begin with the same
// pool segment (equal pre_off) share it: the longest cached prefix of that
// segment, up to the longest member's segment length p_max, is computed
// once per window on every holder of its first block (by the request that
// claimed the group, its leader), and every member derives its own hit: a
// member with segment length p has hit H on an instance whose walk of the
// shared segment stopped at H < p; otherwise its first p blocks are all
// cached there and its own walk resumes at its tail.
constexpr int32_t kGroupMin = 8;             // shortest shared segment walked as a group
constexpr uint32_t kGroupHold = 16;          // holders of the first block per group record
constexpr uint32_t kGroupNone = 0xFFFFFFFFu; // record without a result (more holders)
constexpr int kGroupGenShift = 40;           // key = gen << 40 | (pre_off + 1)
constexpr uint64_t kGroupGenMax = (1ull << 24) - 1;
constexpr int32_t kGroupMaxReq = 1 << 22;    // larger windows are scored without groups

// Record of one group slot: GroupMeta, then up to kGroupHold holders in
// ascending id order as {instance id, hit of the leader's segment there},
// then one word {class, bitmap} for popular groups (below).
struct alignas(8) GroupMeta {
  int32_t plen;  // length of the segment the leader walked
  uint32_t cnt;  // holders of its first block, or kGroupNone
};
constexpr int kGroupRec = 2 + (int)kGroupHold;  // 8-byte words per slot record
// Popular groups (kGroupPop) whose holders all have one hit H* but for at
// most kGroupHold exceptions: the record keeps the exceptions in place of
// the holders and, in its last word, {n_exc << 24 | H*, the first block's
// holder bitmap number}; otherwise that word's first half is kGroupNone.
constexpr int kGroupClsWord = 1 + (int)kGroupHold;
// Class word .y of a popular group that the popular pass's list had no
// room for (the walk pass takes it); a listed one holds its bitmap number.
constexpr uint32_t kGroupUnlisted = 0xFFFFFFFFu;

constexpr uint32_t kGroupLead = 0x80000000u;  // slot_of flag of the group's leader
constexpr uint32_t kGroupNoSlot = 0xFFFFFFFFu;
// GroupMeta.cnt with this bit (and not kGroupNone): the group's first block
// has more holders than a record keeps; the hits of all of them are in the
// popular area, row (cnt & ~kGroupPop).
constexpr uint32_t kGroupPop = 0x80000000u;
constexpr size_t kGroupPopBytes = (size_t)64 << 20;  // popular area: hits of n_inst u32 per row
// Header of the popular area: the first line holds the rows-taken and
// deferral words, then two sets (window parities) of kXcds leader lists'
// {length, longest leader segment}, each pair on a 128-byte line of its own
// (a wave's atomics on one list do not queue behind the others' on a shared
// line).
constexpr uint32_t kListCtrWords = 32;  // 128 bytes

struct GroupTab {
  unsigned long long* keys;  // slots; a key of another generation is an empty slot
  unsigned long long* plen;  // slots: gen << 40 | p_max (an older generation compares lower)
  uint2* rec;                // slots * kGroupRec words
  uint32_t* slot_of;         // per request: slot (| kGroupLead), or kGroupNoSlot
  uint32_t* pop;             // popular rows: pop_cap * n_inst hits (holders' entries only)
  uint32_t* pop_ctr;         // rows taken in this window, then the deferral word (both
                             // reset by the claim pass)
  uint32_t pop_cap;
  uint32_t mask;             // slots - 1
  uint64_t gen;              // this window's generation, 1 .. kGroupGenMax
  // this window's leaders in kXcds lists (list x at x * lcap), each entry
  // (pre_off + 1) << 24 | slot, with their lengths in lctr[x * kListCtrWords]
  // and their longest segments in the next word; lctr_next: the other window
  // parity's words, cleared here for the next window
  unsigned long long* lists;
  uint32_t* lctr;
  uint32_t* lctr_next;
  uint32_t lcap;
  // walkers the walk pass aims for: with fewer groups than that, each group
  // gets up to kGroupSplitMax waves, wave k walking the k-th part of the
  // segment on each holder, and the record's hits are the minima of the
  // parts' first misses (every new leader sets them to ~0 in the claim pass)
  uint32_t walkers;
  // 1: the popular pass runs beside the walk pass (on pools of at most 64 x
  // kPopWords instances), which then skips every listed group.  The claim
  // pass lists the groups whose first block has a holder bitmap in `plist`
  // ({slot, bitmap number}, plist_cap entries; count in
  // lctr[kPopCountWord], cleared by the previous window's claim pass) and
  // stores per bitmap one of its listed groups, its representative (`rep`:
  // (kGroupGenMax - gen) << 32 | slot; a word with another window's tag is
  // stale; any listed group gives the same outputs).  The prefix kernel walks each
  // representative's segment through the index while more than one holder
  // is live and keeps, per holder, the position where it dropped out (~0:
  // live at the stop, `pre_q`) in row `pre` of the bitmap; the member kernel
  // starts every listed group's walk from that row at the common prefix of
  // its segment and its representative's.  Listed group v takes popular
  // row pop_cap + v (the second half of the area).
  uint32_t pop_pass;
  uint2* plist;
  uint32_t plist_cap;
  unsigned long long* rep;
  uint32_t rep_cap;  // holder bitmaps of the index
  uint32_t* pre;     // rep_cap rows of n_inst entries
  uint32_t* pre_q;   // rep_cap
};
constexpr int32_t kPopWords = 64;       // bitmap words of the largest pool the popular pass takes
constexpr uint32_t kPopCountWord = 2;   // on list 0's line of lctr
constexpr uint32_t kGroupSplitMax = 4;
constexpr int32_t kGroupPartMin = 1024;  // positions per part at least

// One of the pool's 64 largest rooms (descending; pads: room -1).
struct alignas(16) TopRoom {
  int64_t room;
  int32_t id;
  int32_t pad;
};
constexpr int kTopRooms = 64;

struct ScoreArgs {
  Tables t;
  GIndex x;
  GroupTab grp;  // keys == nullptr: no prefix groups in this launch
  const int64_t* room_sorted;  // rooms ascending (eligible count = n - lower_bound(L))
  const uint32_t* order0;      // instance ids by (decoding desc, queued asc, id asc)
  const InstState* inst_key;   // the instances' states in that order
  const int4* lm;              // key order: {longest zero-hit admitted chain (blocks, -1 none), id, D, Q}
  const int32_t* lm1;          // maxima of lm[].x over 64-entry chunks
  // key order, per 64-entry chunk: {least t_iter at L = 0 over the
  // instances with A1 > 1, the same over A1 <= 1 (fp32 bits; +inf for
  // none), largest room (int64; -1 for none)}
  const uint4* csum;
  const InstState* inst;
  const int64_t* room;   // per instance: kv_cap - S if A1 <= b_max, else -1 (eligible iff L <= room)
  const TopRoom* rtop;   // the kTopRooms largest rooms
  const DevModel* model;
  const uint64_t* pool;
  int64_t pool_len;
  const ps_req* reqs;
  int32_t n_req;
  int32_t n_inst;
  ps_result* out;
  uint32_t* sizes;       // optional |A|,|C|,|T| per request
  uint32_t* hits_out;    // probe-all diagnostic: n_req * n_inst
  const int32_t* req_order;  // probe-all: requests taken in this order (nullptr: array order)
  uint16_t* scratch;     // per-wave hit rows when they do not fit LDS
  int32_t batch;         // requests per batch of the scoring kernel
  uint32_t sel;          // the model's selector (host copy, picks the kernels)
  uint32_t* defer_any;   // set when the lean kernel left requests to the general one
  int32_t defer_only;    // general kernel: score only requests marked as left to it
  // Hand-over from the rows scorer (dlist == nullptr: the general kernel
  // reads every request's mark instead): the requests it left, in
  // kDeferLists sub-lists of dcap entries (rows wave w appends to sub-list
  // w % kDeferLists); sub-list q's length in dcnt[q * kDeferStride] (one
  // 128-byte line each, cleared by the claim pass).
  uint32_t* dcnt;
  int32_t* dlist;
  int32_t dcap;
};
constexpr int kDeferLists = 64;
constexpr int kDeferStride = 32;

// Order of the exhaustive probe: requests by descending chain length in
// bins of 256 blocks (chains of 16,128 blocks or more share the first bin),
// then by a hash of the shared segment (256 values); invalid descriptors
// last.  Chunks of 64 consecutive requests of the order go to the XCDs in
// turn.
constexpr int32_t kOrderLenBins = 64;
constexpr int kOrderShift = 8;
constexpr int32_t kOrderHashBins = 256;
constexpr int32_t kOrderAll = kOrderLenBins * kOrderHashBins;
constexpr int32_t kOrderChunk = 64;
constexpr int32_t kXcds = 8;  // workgroups go to the XCDs in turn
constexpr uint32_t kGroupHeadWords = kListCtrWords * (1 + 2 * kXcds);

struct CommitArgs {
  Tables t;
  InstState* inst;
  int64_t* room;
  const DevModel* model;
  const uint64_t* pool;
  const ps_req* reqs;
  const int32_t* order;     // entries grouped by instance, array order kept
  const int32_t* grp_off;   // n_grp + 1
  const int32_t* grp_inst;  // n_grp
  int32_t n_grp;
  uint32_t cap;             // distinct keys allowed per instance
  unsigned long long* dropped;
};

// One launch of the per-arrival scheduler: requests [r0, r1) of the window,
// taken in order by a single workgroup.  `hits` holds every request's hit on
// every instance at the launch's starting state, (r1 - r0) x n_inst; the
// kernel extends them in place where a block committed by an earlier
// request of the launch continues the prefix.
constexpr int kSeqMaxThreads = 256;  // workgroup of the per-arrival scheduler (one wave per SIMD)
constexpr int kSeqWaves = kSeqMaxThreads / 64;
constexpr int kSeqStage = 4096;      // chain blocks staged in LDS per request (32 KiB)
constexpr int kSeqU = 4;             // positions per thread in one sweep or insert step
constexpr uint32_t kExtMax = 128;    // hit extensions swept by the workgroup per request
constexpr int kSeqB = 2;             // instances per thread whose loads are issued together

// Speculative batches of the per-arrival scheduler.  Every request of a
// batch is first scored in parallel (one workgroup each) against the state
// at the batch's start; the scheduler workgroup then takes the batch in
// order and, for each request, re-evaluates only the instances that earlier
// requests of the batch were placed on (at most one per request, so at most
// kSpecBatch): when the speculative result settles the decision against the
// current state, the request is decided from it; otherwise it is scored in
// full.  A speculative result keeps |A|, |C|, |T|, W_min and the first
// members of T and of C in the order of their keys.
constexpr int kSpecBatch = kSeqMaxThreads;  // requests per batch at most (one thread per changed instance)
constexpr int kSpecList = 64;               // members of T (and of C) kept per request
constexpr int kSpecTop = 4;                 // per-thread candidates gathered before the merge

struct alignas(16) SpecEntry {
  uint64_t key;  // the selector's key (T) or the fallback key (C); the id in bits 0..15
  uint32_t w;    // the candidate's recomputation penalty W (fp32 bits)
  uint32_t pad;
};

struct alignas(16) SpecRec {
  uint32_t nA, nC, nT;
  uint32_t wmin;       // W_min over A (fp32 bits)
  uint32_t nLT, nLF;   // entries of lt and lf: the first nLT members of T by key (all of T
                       // when nLT == nT), the first nLF members of C by fallback key
  uint32_t pad[2];
  SpecEntry lt[kSpecList];
  SpecEntry lf[kSpecList];
};

struct SeqArgs {
  Tables t;
  InstState* inst;
  int64_t* room;
  const DevModel* model;
  const uint64_t* pool;
  int64_t pool_len;
  const ps_req* reqs;      // the whole window (r indexes it)
  int32_t r0, r1;
  int32_t n_inst;
  uint32_t* hits;
  const int32_t* forced;   // replay: placement of every request (-1 none); null: Algorithm 1
  ps_result* out;          // whole window
  uint32_t* sizes;         // optional |A|,|C|,|T| (Algorithm 1 only)
  uint32_t cap;            // distinct keys allowed per instance
  unsigned long long* dropped;
  const SpecRec* spec;     // speculative results of requests [r0, r1) (null: none)
  unsigned long long* stats;  // [0] += decisions taken from them, [1] += decisions scored in full
};

struct BuildArgs {
  Tables t;
  const int64_t* blk_off;
  const uint64_t* blk;
  int32_t n_inst;
  int64_t n_blk;
  unsigned long long* full;  // inserts that found no free slot (never for valid caps)
  uint32_t* won;             // n_blk: 1 where this list entry inserted its key
  uint32_t* slot_of;         // n_blk: table slot of the entry's key
  uint32_t* rank;            // n_blk: exclusive scan of `won` (global)
};

}  // namespace ps

// Kernel launchers (ps_kernels.hip).
hipError_t ps_launch_build(const ps::BuildArgs& a, hipStream_t s);  // slots, won, slot_of
hipError_t ps_launch_rows(const ps::BuildArgs& a, hipStream_t s);   // rows, rowpos (needs rank)
hipError_t ps_exclusive_scan_u32(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t s);
// fast: the policy of the four-requests-per-wave scorer (keyed selector,
// monotone model, no TTFT admission, no set sizes) selects a kernel built
// for it alone.
hipError_t ps_launch_score(const ps::ScoreArgs& a, bool hits_in_lds, int grid, bool probe_all,
                           hipStream_t s, bool fast = false);
// Order of the exhaustive probe's requests (bins: kOrderAll words).
hipError_t ps_launch_order(const ps_req* reqs, int32_t n, int64_t pool_len, uint32_t* bins,
                           int32_t* order, hipStream_t s);
// The lean scorer with four requests per wave (rows of 16 lanes), for the
// keyed selectors with a monotone model, no TTFT admission, no candidate-set
// sizes and at most kRowsMaxInst instances; its LDS and resident waves per CU.
constexpr int32_t kRowsMaxInst = 4096;
hipError_t ps_launch_lean_rows(const ps::ScoreArgs& a, int grid, hipStream_t s);
size_t ps_lean_rows_lds_bytes(int32_t n_inst);
int32_t ps_lean_rows_waves_per_cu(int32_t n_inst);
// The general kernel's resident waves per CU.
int32_t ps_score_waves_per_cu(int32_t n_inst, bool hits_in_lds, bool fast);
// Lean scorer (requests with group records); its LDS and resident waves per CU.
hipError_t ps_launch_lean(const ps::ScoreArgs& a, int grid, hipStream_t s);
size_t ps_lean_lds_bytes(int32_t n_inst);
int32_t ps_lean_waves_per_cu(int32_t n_inst);
bool ps_hits_fit_lds(int32_t n_inst);
// Prefix index build (ps_index.hip): from the per-instance tables.  Frees and
// replaces *x.  count_host: distinct keys per instance.
hipError_t ps_build_index(const ps::Tables& t, int32_t n_inst, const uint32_t* count_host,
                          ps::GIndex* x, hipStream_t s);
void ps_free_index(ps::GIndex* x);
hipError_t ps_launch_commit(const ps::CommitArgs& a, hipStream_t s);
// Zero-hit admission thresholds in key order and their chunk maxima.
hipError_t ps_launch_lmax(const ps::InstState* inst_key, const uint32_t* order0,
                          const ps::DevModel* m, int32_t n, int4* lm, int32_t* lm1, uint4* csum,
                          hipStream_t s);
// Prefix groups of a window: slot of every request and the longest member
// segment per group, then the walks of the leaders.
// grid: a multiple of 64; mid (optional) is recorded between the claim and
// walk launches
// aux, fork, join: with a.grp.pop_pass, the second stream the walk pass
// runs on beside the popular pass (on s), and the events of the fork and
// join.
hipError_t ps_launch_group(const ps::ScoreArgs& a, int grid, hipStream_t s, hipEvent_t mid,
                           hipStream_t aux = nullptr, hipEvent_t fork = nullptr,
                           hipEvent_t join = nullptr);
// Per-arrival scheduler: one workgroup of `threads` (a multiple of 64, at
// most kSeqMaxThreads) over requests [a.r0, a.r1).
hipError_t ps_launch_seq(const ps::SeqArgs& a, int threads, hipStream_t s);
// Speculative scoring of requests [a.r0, a.r1) (one workgroup each) into
// out[r - a.r0]; a.hits holds their hits at the current state.
hipError_t ps_launch_spec(const ps::SeqArgs& a, ps::SpecRec* out, hipStream_t s);
size_t ps_seq_lds_bytes(int32_t n_inst);
size_t ps_score_lds_bytes(int32_t n_inst);
// Pools small enough for the scoring kernel to keep rooms, states and
// zero-hit thresholds in LDS (it then runs a persistent grid).
bool ps_score_small(int32_t n_inst);
// Requests per batch of the scoring kernel (one wave loads a batch's
// inputs together): about one batch per resident wave, at most 4.
int32_t ps_score_batch(int32_t n_req, int32_t resident_waves);
