// Host side of the C ABI declared in include/packserve.h: argument checks,
// device memory, streams and kernel launches.  Every step of the scoring
// path runs in the kernels of ps_kernels.hip; nothing here computes a
// decision.

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ps_device.h"

using namespace ps;

namespace {

thread_local std::string g_create_error;

// Waves of the persistent scoring grid (per CU) when hit rows live in
// device scratch instead of LDS.
constexpr int kScratchRowsPerCU = 16;

// Scoring calls whose launches are timed between two reads of the timing.
constexpr int32_t kTimingCalls = 4096;
// Events per timed call: around the claim pass, the group walk, the lean
// scorer and the general scorer.
constexpr int kTimingEvents = 5;

// Entries per leader list for a window of n_req requests: the claim pass's
// waves (4 per 256 requests) take the kXcds lists in turn, at most 64
// leaders per wave.
constexpr uint32_t leader_list_cap(int32_t n_req) {
  return ((uint32_t)((n_req + 255) / 256) * 4u + kXcds - 1) / kXcds * 64u;
}

// The fixed scratch of the allocation-free scoring entry point: one window's
// prefix-group table for up to kFixedMaxReq requests, laid out as the
// context's own (slot keys and tagged lengths, slot records, per-request
// slots, leader lists, counter words, popular rows).
constexpr int32_t kFixedMaxReq = 65536;
constexpr uint32_t kFixedSlots = 131072;  // a power of two >= 2 * kFixedMaxReq
constexpr uint32_t kFixedListCap = leader_list_cap(kFixedMaxReq);
constexpr size_t kFixedPopBytes = (size_t)16 << 20;
constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr size_t kFixedOffKeys = 0;
constexpr size_t kFixedOffRec = align256(kFixedOffKeys + 2 * (size_t)kFixedSlots * sizeof(unsigned long long));
constexpr size_t kFixedOffSlot = align256(kFixedOffRec + (size_t)kFixedSlots * kGroupRec * sizeof(uint2));
constexpr size_t kFixedOffList = align256(kFixedOffSlot + (size_t)kFixedMaxReq * sizeof(uint32_t));
constexpr size_t kFixedOffHead = align256(kFixedOffList + (size_t)kXcds * kFixedListCap * sizeof(unsigned long long));
constexpr size_t kFixedOffPop = align256(kFixedOffHead + (size_t)kGroupHeadWords * sizeof(uint32_t));
constexpr size_t kFixedBytes = align256(kFixedOffPop + kFixedPopBytes);  // about 37 MiB
static_assert(kFixedSlots >= 2u * (uint32_t)kFixedMaxReq, "fixed group table too small");

}  // namespace

// The allocation-free entry point's device scratch: one copy per GPU, held
// until the process ends.  Host code never passes this name to a kernel or a
// copy: it uses the address hipGetSymbolAddress returned for the device.
static __device__ __align__(256) unsigned char scratch[kFixedBytes];

namespace {

// Per device: the address of `scratch` on that device (set once, at the
// first ps_create on it) and the window generation of its group table.
struct FixedScratch {
  unsigned char* ptr = nullptr;
  uint64_t gen = 0;
};
constexpr int kMaxDevices = 64;
std::mutex g_fixed_mu;
FixedScratch g_fixed[kMaxDevices];

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Zeroes n 32-bit words with a kernel (not a memset node, so a caller may
// capture it in a graph).
hipError_t fill_zero(void* p, size_t words, hipStream_t s) {
  const int grid = (int)std::min<size_t>((words + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_u32_kernel, dim3(grid), dim3(256), 0, s, (uint32_t*)p, words, 0u);
  return hipGetLastError();
}

// What must start at zero in the fixed group table: the slot keys and
// tagged lengths (a zero key is an empty slot) and the counter words.
hipError_t clear_fixed(unsigned char* base, hipStream_t s) {
  hipError_t e = fill_zero(base + kFixedOffKeys, 2 * (size_t)kFixedSlots * 2, s);
  if (e == hipSuccess) e = fill_zero(base + kFixedOffHead, kGroupHeadWords, s);
  return e;
}

}  // namespace

struct ps_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  // the scoring call's second stream (the walk pass, beside the popular
  // pass on the calling stream) and the events of its fork and join
  hipStream_t aux = nullptr;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  int num_cus = 0;
  std::string err;
  bool loaded = false;
  // snapshot
  int32_t n_inst = 0;
  int32_t cap = 0;
  Tables t{};
  InstState* d_inst = nullptr;
  int64_t* d_room = nullptr;
  int64_t* d_room_sorted = nullptr;
  uint32_t* d_order0 = nullptr;
  InstState* d_inst_key = nullptr;  // states in d_order0's order
  TopRoom* d_rtop = nullptr;         // the kTopRooms largest rooms with their ids
  int32_t lean_wpc = 0;              // resident lean-scorer waves per CU (0: not asked yet)
  int32_t rows_wpc = 0;              // the same for the four-requests-per-wave scorer
  int32_t score_wpc = 0;             // the same for the general scorer (fast policy)
  int4* d_lm = nullptr;              // zero-hit admission thresholds in that order
  int32_t* d_lm1 = nullptr;          // their maxima per 64 positions
  uint4* d_csum = nullptr;           // per 64 positions: least t_iter (A1 > 1, A1 <= 1), largest room
  GIndex x{nullptr, nullptr, nullptr, 0, 0, 64};
  DevModel* d_model = nullptr;
  unsigned long long* d_counter = nullptr;
  uint16_t* d_scratch = nullptr;
  int scratch_rows = 0;
  bool hits_in_lds = true;
  std::vector<InstState> h_state;
  std::vector<uint32_t> h_count;
  DevModel h_model{};
  // feedback: EMA factors in double between updates; recent output lengths
  std::vector<double> gamma64;
  std::vector<int32_t> lout_ring;
  int64_t lout_seen = 0;
  float lout_raw = 0.0f;
  // staging for the host-memory entry points
  void* d_stage[3] = {nullptr, nullptr, nullptr};
  size_t stage_cap[3] = {0, 0, 0};
  // per-arrival scheduler: hits of one launch's requests on every instance
  uint32_t* d_seq_hits = nullptr;
  size_t seq_hits_cap = 0;  // elements
  size_t seq_budget = (size_t)256 << 20;  // bytes of hits per scheduler launch
  // speculative batches (requests per batch; 0: every request scored in full)
  int32_t spec_batch = kSpecBatch;
  SpecRec* d_spec = nullptr;
  int32_t spec_cap = 0;                          // records
  unsigned long long* d_seq_stats = nullptr;     // decisions from speculation, scored in full
  // prefix groups of the scored windows: slot keys (tagged with a window
  // generation, so a new window needs no clearing), slot records, and each
  // request's slot
  unsigned long long* d_gkeys = nullptr;  // keys, then the tagged segment lengths
  uint2* d_grec = nullptr;
  uint32_t* d_gslot = nullptr;
  uint32_t* d_gpop = nullptr;  // kGroupHeadWords counter words (rows taken, deferral; two sets
                               // of leader list lengths, one 128-byte line per list), then
                               // the popular rows
  unsigned long long* d_glist = nullptr;  // the leaders' lists (kXcds * glcap)
  uint32_t glcap = 0;           // entries per list
  uint32_t gslots = 0;   // power of two
  int32_t greq_cap = 0;  // entries of d_gslot
  // the rows scorer's hand-over: kDeferLists sub-list lengths (one 128-byte
  // line each) and the sub-lists (dcap entries each)
  uint32_t* d_dcnt = nullptr;
  int32_t* d_dlist = nullptr;
  int64_t dcap = 0;
  uint64_t ggen = 0;
  uint2* d_gplist = nullptr;  // the popular pass's groups
  uint32_t gplist_cap = 0;
  unsigned long long* d_grep = nullptr;  // representatives, per holder bitmap
  uint32_t grep_cap = 0;
  uint32_t* d_gpre = nullptr;            // prefix rows (grep_cap x n_inst), then grep_cap ends
  size_t gpre_cap = 0;                   // words
  // order of the exhaustive probe's requests (counting-sort bins, order)
  uint32_t* d_obins = nullptr;
  int32_t* d_order = nullptr;
  int32_t order_cap = 0;
  // optional per-launch timing of the scoring path: events recorded on the
  // call's stream before the group pass, between it and the scoring kernel,
  // and after it, for up to kTimingCalls calls
  bool timing = false;
  int32_t n_timed = 0;
  std::vector<hipEvent_t> ev;  // 3 per call
};

namespace {

ps_status fail(ps_ctx* c, ps_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  else g_create_error = buf;
  return code;
}

#define HIP_TRY(ctx, call)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(ctx, e_ == hipErrorOutOfMemory ? PS_E_NOMEM : PS_E_DEVICE, "%s: %s", #call, \
                  hipGetErrorString(e_));                                                   \
  } while (0)

// Makes ctx's device current for the scope of an entry point.
struct DeviceScope {
  int prev = -1;
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceScope() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

template <class T>
void dfree(T*& p) {
  if (p) (void)hipFree((void*)p);
  p = nullptr;
}

// Grows staging buffer k to at least `bytes`.
ps_status stage_buffer(ps_ctx* c, int k, size_t bytes, void** out) {
  if (bytes > c->stage_cap[k]) {
    if (c->d_stage[k]) (void)hipFree(c->d_stage[k]);
    c->d_stage[k] = nullptr;
    c->stage_cap[k] = 0;
    size_t want = std::max(bytes, (size_t)4096);
    HIP_TRY(c, hipMalloc(&c->d_stage[k], want));
    c->stage_cap[k] = want;
  }
  *out = c->d_stage[k];
  return PS_OK;
}

int32_t segment_of_host(const ps_model& m, int32_t B) {
  for (int32_t s = 0; s < m.n_seg; ++s)
    if (B <= m.seg_ub[s]) return s;
  return m.n_seg - 1;
}

bool finite(float x) { return std::isfinite(x); }

ps_status check_model(ps_ctx* c, const ps_model* m) {
  if (!m) return fail(c, PS_E_INVAL, "model is NULL");
  if (m->n_seg < 1 || m->n_seg > PS_MAX_SEG)
    return fail(c, PS_E_RANGE, "n_seg %d outside [1, %d]", m->n_seg, PS_MAX_SEG);
  for (int k = 0; k < 6; ++k)
    if (!finite(m->alpha[k])) return fail(c, PS_E_INVAL, "alpha[%d] is not finite", k);
  for (int s = 0; s < m->n_seg; ++s) {
    if (m->seg_ub[s] < 1 || (s > 0 && m->seg_ub[s] <= m->seg_ub[s - 1]))
      return fail(c, PS_E_INVAL, "seg_ub must be positive and strictly ascending (segment %d)", s);
    for (int k = 0; k < 3; ++k)
      if (!finite(m->beta[s][k])) return fail(c, PS_E_INVAL, "beta[%d][%d] is not finite", s, k);
    if (!finite(m->gamma[s]) || !(m->gamma[s] > 0.0f))
      return fail(c, PS_E_INVAL, "gamma[%d] must be finite and > 0", s);
  }
  if (!finite(m->eta) || m->eta < 0.0f) return fail(c, PS_E_INVAL, "eta must be finite and >= 0");
  if (!finite(m->tpot_slo) || m->tpot_slo < 0.0f)
    return fail(c, PS_E_INVAL, "tpot_slo must be finite and >= 0");
  if (!finite(m->ttft_floor) || m->ttft_floor < 0.0f)
    return fail(c, PS_E_INVAL, "ttft_floor must be finite and >= 0");
  if (!finite(m->lout) || m->lout < 0.0f) return fail(c, PS_E_INVAL, "lout must be finite and >= 0");
  if (m->block_tokens < 1 || m->block_tokens > PS_MAX_BLOCK_TOKENS)
    return fail(c, PS_E_RANGE, "block_tokens %d outside [1, %d]", m->block_tokens, PS_MAX_BLOCK_TOKENS);
  if (m->b_max < 1 || m->b_max > PS_MAX_BATCH)
    return fail(c, PS_E_RANGE, "b_max %d outside [1, %d]", m->b_max, PS_MAX_BATCH);
  if (m->kv_cap_tokens < 0) return fail(c, PS_E_RANGE, "kv_cap_tokens is negative");
  if (m->flags & ~(PS_F_TTFT_ADMIT | PS_F_NO_KVC_FILTER | PS_F_NO_TPOT_FILTER | PS_F_FALLBACK_DCQ |
                   PS_F_SELECTOR(0xF)))
    return fail(c, PS_E_INVAL, "unknown flag bits 0x%x", m->flags);
  if (((m->flags >> 8) & 0xF) > PS_SEL_LMETRIC)
    return fail(c, PS_E_INVAL, "unknown selector %u", (m->flags >> 8) & 0xF);
  return PS_OK;
}

// Whether the zero-hit TPOT test of every instance is one threshold on the
// request length L: T_pf(L, 0) = a0 + L (a1 + a3 L) and the decode term
// gamma (b0 + b1 B + b2 (S + L)) are then non-decreasing in L in fp32 too
// (each rounded step is a monotone function of non-negative operands).
uint32_t monotone(const DevModel& d) {
  for (int k = 0; k < 6; ++k)
    if (!std::isfinite(d.a[k])) return 0u;
  if (!(d.a[1] >= 0.0f) || !(d.a[3] >= 0.0f)) return 0u;
  if (!std::isfinite(d.lout1) || !(d.lout1 > 0.0f) || !std::isfinite(d.tau)) return 0u;
  for (int s = 0; s < d.n_seg; ++s) {
    for (int k = 0; k < 4; ++k)
      if (!std::isfinite(d.seg[s][k])) return 0u;
    if (!(d.seg[s][2] >= 0.0f) || !(d.seg[s][3] >= 0.0f)) return 0u;
  }
  return 1u;
}

DevModel device_model(const ps_model& m) {
  DevModel d{};
  for (int k = 0; k < 6; ++k) d.a[k] = m.alpha[k];
  const double a1 = m.alpha[1], a2 = m.alpha[2], a3 = m.alpha[3], a4 = m.alpha[4], a5 = m.alpha[5];
  d.k1 = (float)(a1 - a4);
  d.k2 = (float)(a2 - 2.0 * a5);
  d.k3 = (float)(a3 - a2 + a5);
  d.eta = m.eta;
  d.tau = m.tpot_slo;
  d.ttft_floor = m.ttft_floor;
  d.lout1 = std::max(1.0f, m.lout);
  d.bs = m.block_tokens;
  d.b_max = m.b_max;
  d.kv_cap = m.kv_cap_tokens;
  d.flags = m.flags & 0xFFu;
  d.sel = (m.flags >> 8) & 0xFu;
  d.rand_seed = m.rand_seed;
  d.n_seg = m.n_seg;
  for (int s = 0; s < PS_MAX_SEG; ++s) {
    d.seg_ub[s] = s < m.n_seg ? m.seg_ub[s] : 0;
    for (int k = 0; k < 3; ++k) d.seg[s][k] = s < m.n_seg ? m.beta[s][k] : 0.0f;
    d.seg[s][3] = s < m.n_seg ? m.gamma[s] : 1.0f;
  }
  d.mono = monotone(d);
  return d;
}

ps_status check_reqs_host(ps_ctx* c, const uint64_t* pool, int64_t pool_len, const ps_req* reqs,
                          int32_t n) {
  if (pool_len < 0) return fail(c, PS_E_INVAL, "pool_len is negative");
  if (n > 0 && !reqs) return fail(c, PS_E_INVAL, "reqs is NULL");
  if (pool_len > 0 && !pool) return fail(c, PS_E_INVAL, "pool is NULL");
  for (int32_t r = 0; r < n; ++r) {
    const ps_req& q = reqs[r];
    if (q.pre_len < 0 || q.tail_len < 0 || q.pre_off < 0 || q.tail_off < 0 ||
        q.pre_off > pool_len || q.tail_off > pool_len || q.pre_len > pool_len - q.pre_off ||
        q.tail_len > pool_len - q.tail_off)
      return fail(c, PS_E_RANGE, "request %d lies outside the pool", r);
    if ((int64_t)q.pre_len + q.tail_len > PS_MAX_CHAIN)
      return fail(c, PS_E_RANGE, "request %d chain longer than %d blocks", r, PS_MAX_CHAIN);
  }
  for (int64_t k = 0; k < pool_len; ++k)
    if (pool[k] == 0) return fail(c, PS_E_INVAL, "zero block hash at pool[%lld]", (long long)k);
  return PS_OK;
}

void free_snapshot(ps_ctx* c) {
  dfree(c->t.keys);
  dfree(c->t.count);
  dfree(c->t.rows);
  dfree(c->t.rowpos);
  dfree(c->d_inst);
  dfree(c->d_room);
  dfree(c->d_room_sorted);
  dfree(c->d_order0);
  dfree(c->d_inst_key);
  dfree(c->d_rtop);
  dfree(c->d_lm);
  dfree(c->d_lm1);
  dfree(c->d_csum);
  dfree(c->d_scratch);
  ps_free_index(&c->x);
  c->loaded = false;
}

// Zero-hit admission thresholds for the current state and model, complete
// before the entry point returns.
ps_status refresh_lmax(ps_ctx* c) {
  HIP_TRY(c, ps_launch_lmax(c->d_inst_key, c->d_order0, c->d_model, c->n_inst, c->d_lm, c->d_lm1,
                            c->d_csum, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return PS_OK;
}

// The kTopRooms largest rooms with their ids, descending (pads: room -1).
std::vector<TopRoom> top_rooms(const std::vector<int64_t>& room) {
  std::vector<TopRoom> t(room.size());
  for (size_t i = 0; i < room.size(); ++i) t[i] = TopRoom{room[i], (int32_t)i, 0};
  const size_t k = std::min(room.size(), (size_t)kTopRooms);
  std::partial_sort(t.begin(), t.begin() + (long)k, t.end(),
                    [](const TopRoom& x, const TopRoom& y) { return x.room > y.room; });
  t.resize(kTopRooms, TopRoom{-1, 0, 0});
  return t;
}

// Per-instance room (kv_cap - S when A + 1 <= B_max, else -1; an instance
// is capacity-eligible for a request of L tokens iff L <= room) and the same
// values sorted ascending, so |A| is one binary search.
std::vector<int64_t> rooms_of(const std::vector<InstState>& hs, const DevModel& m) {
  std::vector<int64_t> r(hs.size());
  for (size_t i = 0; i < hs.size(); ++i) r[i] = hs[i].A1 <= m.b_max ? m.kv_cap - hs[i].S : -1;
  return r;
}

int32_t segment_of_dev(const DevModel& m, int32_t B) {
  for (int32_t s = 0; s < m.n_seg; ++s)
    if (B <= m.seg_ub[s]) return s;
  return m.n_seg - 1;
}

// Instance ids in the order of the packing key of a candidate with no cached
// prefix: most decoding first, then fewest queued, then lowest id.
std::vector<InstState> states_in_order(const std::vector<InstState>& hs,
                                       const std::vector<uint32_t>& order) {
  std::vector<InstState> v(order.size());
  for (size_t k = 0; k < order.size(); ++k) v[k] = hs[order[k]];
  return v;
}

std::vector<uint32_t> key_order(const std::vector<InstState>& hs) {
  std::vector<uint32_t> o(hs.size());
  for (size_t i = 0; i < o.size(); ++i) o[i] = (uint32_t)i;
  std::sort(o.begin(), o.end(), [&](uint32_t x, uint32_t y) {
    if (hs[x].D != hs[y].D) return hs[x].D > hs[y].D;
    if (hs[x].Q != hs[y].Q) return hs[x].Q < hs[y].Q;
    return x < y;
  });
  return o;
}

// Upload the host copy of the instance state and everything derived from it
// (rooms, sorted rooms, key order).
ps_status refresh_derived(ps_ctx* c) {
  for (InstState& st : c->h_state) {
    st.A1 = st.D + st.Q + 1;
    st.seg = segment_of_dev(c->h_model, st.A1);
  }
  const std::vector<int64_t> room = rooms_of(c->h_state, c->h_model);
  std::vector<int64_t> rs = room;
  std::sort(rs.begin(), rs.end());
  const std::vector<uint32_t> o0 = key_order(c->h_state);
  HIP_TRY(c, hipMemcpy(c->d_inst, c->h_state.data(), c->h_state.size() * sizeof(InstState),
                       hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemcpy(c->d_room, room.data(), room.size() * sizeof(int64_t), hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemcpy(c->d_room_sorted, rs.data(), rs.size() * sizeof(int64_t), hipMemcpyHostToDevice));
  const std::vector<TopRoom> tr = top_rooms(room);
  HIP_TRY(c, hipMemcpy(c->d_rtop, tr.data(), tr.size() * sizeof(TopRoom), hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemcpy(c->d_order0, o0.data(), o0.size() * sizeof(uint32_t), hipMemcpyHostToDevice));
  const std::vector<InstState> ik = states_in_order(c->h_state, o0);
  HIP_TRY(c, hipMemcpy(c->d_inst_key, ik.data(), ik.size() * sizeof(InstState), hipMemcpyHostToDevice));
  return refresh_lmax(c);
}

ps_status upload_model(ps_ctx* c) {
  c->h_model.mono = monotone(c->h_model);
  HIP_TRY(c, hipMemcpy(c->d_model, &c->h_model, sizeof c->h_model, hipMemcpyHostToDevice));
  return refresh_lmax(c);
}

}  // namespace

extern "C" {

ps_status ps_create(int device, ps_ctx** out) {
  if (!out) return fail(nullptr, PS_E_INVAL, "out is NULL");
  *out = nullptr;
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess)
    return fail(nullptr, PS_E_DEVICE, "hipGetDeviceCount: %s", hipGetErrorString(e));
  if (device < 0 || device >= n)
    return fail(nullptr, PS_E_INVAL, "device %d outside [0, %d)", device, n);
  ps_ctx* c = new (std::nothrow) ps_ctx();
  if (!c) return fail(nullptr, PS_E_NOMEM, "host allocation failed");
  c->device = device;
  DeviceScope ds(device);
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->aux, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->fork_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->join_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipMalloc((void**)&c->d_model, sizeof(DevModel));
  if (e == hipSuccess) e = hipMalloc((void**)&c->d_counter, sizeof(unsigned long long));
  if (e != hipSuccess) {
    ps_destroy(c);
    return fail(nullptr, PS_E_DEVICE, "device set-up failed: %s", hipGetErrorString(e));
  }
  c->num_cus = prop.multiProcessorCount;
  // Once per device, with the device current: the address of the fixed
  // scratch on this device, cleared where it must start at zero.
  if (device < kMaxDevices) {
    std::lock_guard<std::mutex> lk(g_fixed_mu);
    if (!g_fixed[device].ptr) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e == hipSuccess) e = clear_fixed((unsigned char*)p, c->stream);
      if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
      if (e != hipSuccess) {
        ps_destroy(c);
        return fail(nullptr, PS_E_DEVICE, "fixed scratch set-up failed: %s", hipGetErrorString(e));
      }
      g_fixed[device].ptr = (unsigned char*)p;
    }
  }
  *out = c;
  return PS_OK;
}

ps_status ps_destroy(ps_ctx* c) {
  if (!c) return PS_OK;
  DeviceScope ds(c->device);
  if (c->stream) (void)hipStreamSynchronize(c->stream);
  if (c->aux) (void)hipStreamSynchronize(c->aux);
  free_snapshot(c);
  dfree(c->d_model);
  dfree(c->d_counter);
  for (int k = 0; k < 3; ++k)
    if (c->d_stage[k]) (void)hipFree(c->d_stage[k]);
  dfree(c->d_seq_hits);
  dfree(c->d_spec);
  dfree(c->d_seq_stats);
  dfree(c->d_gkeys);
  dfree(c->d_grec);
  dfree(c->d_gslot);
  dfree(c->d_dcnt);
  dfree(c->d_dlist);
  dfree(c->d_gpop);
  dfree(c->d_glist);
  dfree(c->d_gplist);
  dfree(c->d_grep);
  dfree(c->d_gpre);
  dfree(c->d_obins);
  dfree(c->d_order);
  for (hipEvent_t e : c->ev) (void)hipEventDestroy(e);
  if (c->stream) (void)hipStreamDestroy(c->stream);
  if (c->aux) (void)hipStreamDestroy(c->aux);
  if (c->fork_ev) (void)hipEventDestroy(c->fork_ev);
  if (c->join_ev) (void)hipEventDestroy(c->join_ev);
  delete c;
  return PS_OK;
}

const char* ps_last_error(const ps_ctx* c) {
  return c ? c->err.c_str() : g_create_error.c_str();
}

#ifndef PS_SOURCE_HASH
#define PS_SOURCE_HASH "unknown"
#endif
const char* ps_build_id(void) { return PS_SOURCE_HASH; }

ps_status ps_load_instances(ps_ctx* c, const ps_instances* in, const ps_model* m) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!in) return fail(c, PS_E_INVAL, "instances is NULL");
  ps_status st = check_model(c, m);
  if (st != PS_OK) return st;
  const int32_t n = in->n_inst;
  if (n < 1 || n > PS_MAX_INST) return fail(c, PS_E_RANGE, "n_inst %d outside [1, %d]", n, PS_MAX_INST);
  if (in->table_cap_blocks < 1 || in->table_cap_blocks > PS_MAX_TABLE_CAP)
    return fail(c, PS_E_RANGE, "table_cap_blocks %d outside [1, %d]", in->table_cap_blocks,
                PS_MAX_TABLE_CAP);
  if (!in->blk_off || !in->decoding || !in->queued || !in->pending_tok || !in->ctx_tok)
    return fail(c, PS_E_INVAL, "instance array is NULL");
  if (in->blk_off[0] != 0) return fail(c, PS_E_INVAL, "blk_off[0] must be 0");
  for (int32_t i = 0; i < n; ++i) {
    const int64_t len = in->blk_off[i + 1] - in->blk_off[i];
    if (len < 0) return fail(c, PS_E_INVAL, "blk_off not ascending at instance %d", i);
    if (len > in->table_cap_blocks)
      return fail(c, PS_E_RANGE, "instance %d lists %lld blocks > table_cap_blocks %d", i,
                  (long long)len, in->table_cap_blocks);
    if (in->decoding[i] < 0 || in->decoding[i] > PS_MAX_DQ || in->queued[i] < 0 ||
        in->queued[i] > PS_MAX_DQ)
      return fail(c, PS_E_RANGE, "instance %d: decoding/queued outside [0, %d]", i, PS_MAX_DQ);
    if (in->pending_tok[i] < 0 || in->pending_tok[i] > PS_MAX_PENDING)
      return fail(c, PS_E_RANGE, "instance %d: pending_tok outside [0, 2^34]", i);
    if (in->ctx_tok[i] < 0 || in->ctx_tok[i] > PS_MAX_CONTEXT)
      return fail(c, PS_E_RANGE, "instance %d: ctx_tok outside [0, 2^46]", i);
  }
  const int64_t n_blk = in->blk_off[n];
  if (n_blk > 0 && !in->blk) return fail(c, PS_E_INVAL, "blk is NULL");
  for (int64_t k = 0; k < n_blk; ++k)
    if (in->blk[k] == 0) return fail(c, PS_E_INVAL, "zero block hash at blk[%lld]", (long long)k);

  // geometry: >= 2 * cap slots, power of two buckets of 8 slots
  int64_t slots = 8;
  while (slots < 2 * (int64_t)in->table_cap_blocks) slots <<= 1;
  const int64_t buckets = slots / kSlotsPerBucket;
  int log2b = 0;
  while ((1ll << log2b) < buckets) ++log2b;

  DeviceScope ds(c->device);
  ps_ctx fresh;  // new device buffers; swapped in only on success
  fresh.t.slots = slots;
  fresh.t.row_cap = in->table_cap_blocks;
  fresh.t.bmask = (uint32_t)(buckets - 1);
  fresh.t.shift = (uint32_t)(64 - log2b);
  const size_t tab_bytes = (size_t)n * (size_t)slots * sizeof(uint64_t);
  const bool lds = ps_hits_fit_lds(n);
  const int rows = lds ? 0 : std::max(1, c->num_cus * kScratchRowsPerCU);
  int64_t* d_off = nullptr;
  uint64_t* d_blk = nullptr;
  uint32_t *d_won = nullptr, *d_slot = nullptr, *d_rank = nullptr;
  auto free_build_temps = [&]() {
    dfree(d_off);
    dfree(d_blk);
    dfree(d_won);
    dfree(d_slot);
    dfree(d_rank);
  };
  auto cleanup = [&]() {
    free_build_temps();
    dfree(fresh.t.keys);
    dfree(fresh.t.count);
    dfree(fresh.t.rows);
    dfree(fresh.t.rowpos);
    dfree(fresh.d_inst);
    dfree(fresh.d_room);
    dfree(fresh.d_room_sorted);
    dfree(fresh.d_order0);
    dfree(fresh.d_inst_key);
    dfree(fresh.d_rtop);
    dfree(fresh.d_lm);
    dfree(fresh.d_lm1);
    dfree(fresh.d_csum);
    dfree(fresh.d_scratch);
    ps_free_index(&fresh.x);
    dfree(d_off);
    dfree(d_blk);
  };
  hipError_t e = hipMalloc((void**)&fresh.t.keys, tab_bytes);
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.t.count, (size_t)n * sizeof(uint32_t));
  if (e == hipSuccess)
    e = hipMalloc((void**)&fresh.t.rowpos, (size_t)n * (size_t)slots * sizeof(uint32_t));
  if (e == hipSuccess)
    e = hipMalloc((void**)&fresh.t.rows, (size_t)n * (size_t)fresh.t.row_cap * sizeof(uint64_t));
  if (e == hipSuccess && n_blk) e = hipMalloc((void**)&d_won, (size_t)n_blk * sizeof(uint32_t));
  if (e == hipSuccess && n_blk) e = hipMalloc((void**)&d_slot, (size_t)n_blk * sizeof(uint32_t));
  if (e == hipSuccess && n_blk) e = hipMalloc((void**)&d_rank, (size_t)n_blk * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_inst, (size_t)n * sizeof(InstState));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_room, (size_t)n * sizeof(int64_t));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_room_sorted, (size_t)n * sizeof(int64_t));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_order0, (size_t)n * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_inst_key, (size_t)n * sizeof(InstState));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_rtop, (size_t)kTopRooms * sizeof(TopRoom));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_lm, (size_t)n * sizeof(int4));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_lm1, (size_t)((n + 63) / 64) * sizeof(int32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&fresh.d_csum, (size_t)((n + 63) / 64) * sizeof(uint4));
  if (e == hipSuccess && rows)
    e = hipMalloc((void**)&fresh.d_scratch, (size_t)rows * (size_t)n * sizeof(uint16_t));
  if (e == hipSuccess) e = hipMalloc((void**)&d_off, (size_t)(n + 1) * sizeof(int64_t));
  if (e == hipSuccess && n_blk) e = hipMalloc((void**)&d_blk, (size_t)n_blk * sizeof(uint64_t));
  if (e != hipSuccess) {
    cleanup();
    return fail(c, e == hipErrorOutOfMemory ? PS_E_NOMEM : PS_E_DEVICE,
                "allocating %.1f MiB of tables: %s", tab_bytes / 1048576.0, hipGetErrorString(e));
  }
  std::vector<InstState> hs((size_t)n);
  for (int32_t i = 0; i < n; ++i) {
    InstState& s = hs[(size_t)i];
    s.D = in->decoding[i];
    s.Q = in->queued[i];
    s.A1 = s.D + s.Q + 1;
    s.seg = segment_of_host(*m, s.A1);
    s.P = in->pending_tok[i];
    s.S = in->ctx_tok[i];
  }
  const DevModel dm = device_model(*m);
  const std::vector<int64_t> hroom = rooms_of(hs, dm);
  std::vector<int64_t> hroom_sorted = hroom;
  std::sort(hroom_sorted.begin(), hroom_sorted.end());
  const std::vector<uint32_t> horder0 = key_order(hs);
  const std::vector<InstState> hinst_key = states_in_order(hs, horder0);
  hipStream_t sm = c->stream;
  e = hipMemsetAsync(fresh.t.keys, 0, tab_bytes, sm);
  if (e == hipSuccess) e = hipMemsetAsync(fresh.t.count, 0, (size_t)n * sizeof(uint32_t), sm);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_counter, 0, sizeof(unsigned long long), sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(d_off, in->blk_off, (size_t)(n + 1) * sizeof(int64_t), hipMemcpyHostToDevice, sm);
  if (e == hipSuccess && n_blk)
    e = hipMemcpyAsync(d_blk, in->blk, (size_t)n_blk * sizeof(uint64_t), hipMemcpyHostToDevice, sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_inst, hs.data(), hs.size() * sizeof(InstState), hipMemcpyHostToDevice, sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_room, hroom.data(), hroom.size() * sizeof(int64_t), hipMemcpyHostToDevice, sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_room_sorted, hroom_sorted.data(), hroom_sorted.size() * sizeof(int64_t),
                       hipMemcpyHostToDevice, sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_order0, horder0.data(), horder0.size() * sizeof(uint32_t),
                       hipMemcpyHostToDevice, sm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_inst_key, hinst_key.data(), hinst_key.size() * sizeof(InstState),
                       hipMemcpyHostToDevice, sm);
  const std::vector<TopRoom> htop = top_rooms(hroom);
  if (e == hipSuccess)
    e = hipMemcpyAsync(fresh.d_rtop, htop.data(), htop.size() * sizeof(TopRoom), hipMemcpyHostToDevice,
                       sm);
  BuildArgs ba{fresh.t, d_off, d_blk, n, n_blk, c->d_counter, d_won, d_slot, d_rank};
  if (e == hipSuccess) e = ps_launch_build(ba, sm);
  if (e == hipSuccess) e = ps_exclusive_scan_u32(d_won, d_rank, n_blk, sm);
  if (e == hipSuccess) e = ps_launch_rows(ba, sm);
  unsigned long long full = 0;
  if (e == hipSuccess)
    e = hipMemcpyAsync(&full, c->d_counter, sizeof full, hipMemcpyDeviceToHost, sm);
  if (e == hipSuccess) e = hipStreamSynchronize(sm);
  if (e == hipSuccess && full) {
    cleanup();
    return fail(c, PS_E_DEVICE, "table build found no free slot for %llu keys", full);
  }
  std::vector<uint32_t> hc((size_t)n);
  if (e == hipSuccess)
    e = hipMemcpy(hc.data(), fresh.t.count, (size_t)n * sizeof(uint32_t), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = ps_build_index(fresh.t, n, hc.data(), &fresh.x, sm);
  if (e != hipSuccess) {
    cleanup();
    return fail(c, e == hipErrorOutOfMemory ? PS_E_NOMEM : PS_E_DEVICE, "building tables: %s",
                hipGetErrorString(e));
  }
  // The model upload is the last step that can fail; the old snapshot stays
  // intact until here.
  e = hipMemcpy(c->d_model, &dm, sizeof dm, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    cleanup();
    if (c->loaded) (void)hipMemcpy(c->d_model, &c->h_model, sizeof c->h_model, hipMemcpyHostToDevice);
    return fail(c, PS_E_DEVICE, "model upload: %s", hipGetErrorString(e));
  }
  free_build_temps();
  free_snapshot(c);
  c->t = fresh.t;
  c->d_inst = fresh.d_inst;
  c->d_room = fresh.d_room;
  c->d_room_sorted = fresh.d_room_sorted;
  c->d_order0 = fresh.d_order0;
  c->d_inst_key = fresh.d_inst_key;
  c->d_rtop = fresh.d_rtop;
  c->lean_wpc = 0;
  c->rows_wpc = 0;
  c->score_wpc = 0;
  c->d_lm = fresh.d_lm;
  c->d_lm1 = fresh.d_lm1;
  c->d_csum = fresh.d_csum;
  c->x = fresh.x;
  c->d_scratch = fresh.d_scratch;
  c->scratch_rows = rows;
  c->hits_in_lds = lds;
  c->n_inst = n;
  c->cap = in->table_cap_blocks;
  c->h_state = std::move(hs);
  c->h_count = std::move(hc);
  c->h_model = dm;
  c->gamma64.assign((size_t)m->n_seg, 0.0);
  for (int32_t k = 0; k < m->n_seg; ++k) c->gamma64[(size_t)k] = m->gamma[k];
  c->lout_ring.clear();
  c->lout_seen = 0;
  c->lout_raw = m->lout;
  c->loaded = true;
  fresh.t.keys = nullptr;
  fresh.t.count = nullptr;
  fresh.t.rows = nullptr;
  fresh.t.rowpos = nullptr;
  fresh.d_inst = nullptr;
  fresh.d_room = nullptr;
  fresh.d_room_sorted = nullptr;
  fresh.d_order0 = nullptr;
  fresh.d_inst_key = nullptr;
  fresh.d_rtop = nullptr;
  fresh.d_lm = nullptr;
  fresh.d_lm1 = nullptr;
  fresh.d_csum = nullptr;
  fresh.x = GIndex{nullptr, nullptr, nullptr, 0, 0, 64};
  fresh.d_scratch = nullptr;
  const ps_status lst = refresh_lmax(c);
  if (lst != PS_OK) {
    free_snapshot(c);
    return lst;
  }
  return PS_OK;
}

// Groups whose first block has a holder bitmap are walked by the popular
// pass, beside the walk pass, on pools of at most 64 x kPopWords instances
// whose index has such blocks.
static bool popular_pass_ok(const ps_ctx* c) {
  return c->x.n_pop > 0 && c->n_inst <= 64 * kPopWords &&
         (size_t)c->x.n_pop * ((size_t)c->n_inst + 1) * sizeof(uint32_t) <= ((size_t)256 << 20);
}

// Group table for a window of n_req requests (at least two slots per
// request) and the next window generation.  Grows (and clears) only when a
// larger window arrives; a wrapped generation clears the keys once.
static ps_status group_buffers(ps_ctx* c, int32_t n_req, hipStream_t s) {
  uint32_t want = 64;
  while (want < 2u * (uint32_t)n_req) want <<= 1;
  bool clear = false;
  if (want > c->gslots) {
    dfree(c->d_gkeys);
    dfree(c->d_grec);
    c->gslots = 0;
    HIP_TRY(c, hipMalloc((void**)&c->d_gkeys, 2 * (size_t)want * sizeof(unsigned long long)));
    HIP_TRY(c, hipMalloc((void**)&c->d_grec, (size_t)want * kGroupRec * sizeof(uint2)));
    c->gslots = want;
    clear = true;
  }
  if (!c->d_gpop) {
    // two halves of rows: the walk pass's, then the popular pass's
    HIP_TRY(c, hipMalloc((void**)&c->d_gpop, 2 * kGroupPopBytes + kGroupHeadWords * sizeof(uint32_t)));
    HIP_TRY(c, hipMemsetAsync(c->d_gpop, 0, kGroupHeadWords * sizeof(uint32_t), s));  // counter words
  }
  const uint32_t lcap = leader_list_cap(n_req);
  if (lcap > c->glcap) {
    dfree(c->d_glist);
    c->glcap = 0;
    HIP_TRY(c, hipMalloc((void**)&c->d_glist, (size_t)kXcds * lcap * sizeof(unsigned long long)));
    c->glcap = lcap;
  }
  if (n_req > c->greq_cap) {
    dfree(c->d_gslot);
    c->greq_cap = 0;
    HIP_TRY(c, hipMalloc((void**)&c->d_gslot, (size_t)n_req * sizeof(uint32_t)));
    c->greq_cap = n_req;
  }
  // the popular pass lists at most one entry per group: no more than the
  // window's requests, nor than the popular area's rows
  const uint32_t pcap = (uint32_t)std::min<size_t>((size_t)n_req,
                                                   kGroupPopBytes / ((size_t)c->n_inst * sizeof(uint32_t)));
  bool clear_rep = false;
  if (popular_pass_ok(c)) {
    if (pcap > c->gplist_cap) {
      dfree(c->d_gplist);
      c->gplist_cap = 0;
      HIP_TRY(c, hipMalloc((void**)&c->d_gplist, (size_t)pcap * sizeof(uint2)));
      c->gplist_cap = pcap;
    }
    if (c->x.n_pop > c->grep_cap) {
      dfree(c->d_grep);
      c->grep_cap = 0;
      HIP_TRY(c, hipMalloc((void**)&c->d_grep, (size_t)c->x.n_pop * sizeof(unsigned long long)));
      c->grep_cap = c->x.n_pop;
      clear_rep = true;
    }
    const size_t pre_words = (size_t)c->x.n_pop * ((size_t)c->n_inst + 1);
    if (pre_words > c->gpre_cap) {
      dfree(c->d_gpre);
      c->gpre_cap = 0;
      HIP_TRY(c, hipMalloc((void**)&c->d_gpre, pre_words * sizeof(uint32_t)));
      c->gpre_cap = pre_words;
    }
  }
  if (++c->ggen > kGroupGenMax) {
    c->ggen = 1;
    clear = true;
  }
  if (clear) {
    HIP_TRY(c, hipMemsetAsync(c->d_gkeys, 0, 2 * (size_t)c->gslots * sizeof(unsigned long long), s));
    HIP_TRY(c, hipMemsetAsync(c->d_gpop, 0, kGroupHeadWords * sizeof(uint32_t), s));  // list lengths
  }
  if ((clear || clear_rep) && c->grep_cap)  // representatives: all ones is above every tag
    HIP_TRY(c, hipMemsetAsync(c->d_grep, 0xFF, (size_t)c->grep_cap * sizeof(unsigned long long), s));
  return PS_OK;
}

// fixed (optional): the window's prefix-group table in the fixed scratch
// instead of the context's (the allocation-free entry point; no timing).
static ps_status launch_score(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                              const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                              uint32_t* d_sizes, uint32_t* d_hits, hipStream_t s,
                              const GroupTab* fixed = nullptr) {
  ScoreArgs a{};
  a.t = c->t;
  a.x = c->x;
  a.room_sorted = c->d_room_sorted;
  a.order0 = c->d_order0;
  a.inst_key = c->d_inst_key;
  a.rtop = c->d_rtop;
  a.lm = c->d_lm;
  a.lm1 = c->d_lm1;
  a.csum = c->d_csum;
  a.inst = c->d_inst;
  a.room = c->d_room;
  a.model = c->d_model;
  a.pool = d_pool;
  a.pool_len = pool_len;
  a.reqs = d_reqs;
  a.n_req = n_req;
  a.n_inst = c->n_inst;
  a.out = d_out;
  a.sizes = d_sizes;
  a.hits_out = d_hits;
  a.scratch = c->d_scratch;
  a.grp = GroupTab{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0u, 0u, 0ull,
                   nullptr, nullptr, nullptr, 0u, 1u};
  a.sel = c->h_model.sel;
  a.defer_any = nullptr;
  a.defer_only = 0;
  a.dcnt = nullptr;
  a.dlist = nullptr;
  a.dcap = 0;
  a.req_order = nullptr;
  const bool probe_all = d_hits != nullptr;
  if (probe_all) {  // longest chains first
    if (!c->d_obins)
      HIP_TRY(c, hipMalloc((void**)&c->d_obins, kOrderAll * sizeof(uint32_t)));
    if (n_req > c->order_cap) {
      dfree(c->d_order);
      c->order_cap = 0;
      HIP_TRY(c, hipMalloc((void**)&c->d_order, (size_t)n_req * sizeof(int32_t)));
      c->order_cap = n_req;
    }
    HIP_TRY(c, ps_launch_order(d_reqs, n_req, pool_len, c->d_obins, c->d_order, s));
    a.req_order = c->d_order;
  }
  if (!probe_all && fixed) {
    a.grp = *fixed;
    a.defer_any = fixed->pop_ctr + 1;
  } else if (!probe_all && n_req <= kGroupMaxReq && pool_len < ((int64_t)1 << kGroupGenShift) - 1) {
    ps_status st = group_buffers(c, n_req, s);
    if (st != PS_OK) return st;
    a.grp = GroupTab{c->d_gkeys,
                     c->d_gkeys + c->gslots,
                     c->d_grec,
                     c->d_gslot,
                     c->d_gpop + kGroupHeadWords,
                     c->d_gpop,
                     (uint32_t)(kGroupPopBytes / ((size_t)c->n_inst * sizeof(uint32_t))),
                     c->gslots - 1u,
                     c->ggen,
                     c->d_glist,
                     c->d_gpop + kListCtrWords * (1u + kXcds * (uint32_t)(c->ggen & 1u)),
                     c->d_gpop + kListCtrWords * (1u + kXcds * (uint32_t)((c->ggen + 1u) & 1u)),
                     c->glcap,
                     // walkers: half the resident waves (8 per CU)
                     (uint32_t)(8 * c->num_cus),
                     popular_pass_ok(c) && c->gplist_cap ? 1u : 0u,
                     c->d_gplist,
                     c->gplist_cap,
                     c->d_grep,
                     c->x.n_pop,
                     c->d_gpre,
                     c->d_gpre + (size_t)c->x.n_pop * (size_t)c->n_inst};
    a.defer_any = c->d_gpop + 1;
  }
  // The scoring kernel takes batches of a.batch requests per wave; a small
  // pool's waves copy the pool's state into LDS once and take batches in
  // turn (16 waves per CU: 4 per SIMD).  The exhaustive probe takes one
  // request per wave.
  a.batch = ps_score_batch(n_req, c->num_cus * 16);
  const int batches = (n_req + a.batch - 1) / a.batch;
  const int grid = probe_all                       ? (n_req + kXcds * kOrderChunk - 1) / (kXcds * kOrderChunk) * (kXcds * kOrderChunk)
                   : ps_score_small(c->n_inst) ? std::min(batches, c->num_cus * 16)
                   : c->hits_in_lds            ? batches
                                               : std::min(batches, c->scratch_rows);
  // Timed calls record kTimingEvents events: before the claim pass, between
  // it and the group walk, after the walk, after the lean scorer, after the
  // general scorer (a part that is not launched spans no time).
  hipEvent_t* ev = nullptr;
  if (c->timing && !probe_all && !fixed && c->n_timed < kTimingCalls) {
    if (c->ev.size() < kTimingEvents * (size_t)(c->n_timed + 1)) {
      for (int k = 0; k < kTimingEvents; ++k) {
        hipEvent_t e = nullptr;
        HIP_TRY(c, hipEventCreate(&e));
        c->ev.push_back(e);
      }
    }
    ev = &c->ev[kTimingEvents * (size_t)c->n_timed];
  }
  // The lean scorer first when the groups give the requests their hits and
  // the selector is neither Random nor H-C-Q (persistent grid at its own
  // occupancy); the general scorer then finishes what it left.
  const bool lean = !probe_all && a.grp.keys && a.sel != PS_SEL_RANDOM && a.sel != PS_SEL_HCQ;
  const DevModel& hm = c->h_model;
  const bool rows = lean && !d_sizes && hm.mono && !(hm.flags & PS_F_TTFT_ADMIT) &&
                    (a.sel == PS_SEL_DCQ || a.sel == PS_SEL_DQ || a.sel == PS_SEL_DQC) &&
                    c->n_inst <= kRowsMaxInst;
  int rows_grid = 0;
  if (rows) {
    if (!c->rows_wpc) c->rows_wpc = ps_lean_rows_waves_per_cu(c->n_inst);
    const int n_batch = (n_req + 3) / 4;
    rows_grid = std::min(n_batch, c->num_cus * c->rows_wpc);
    if (!fixed) {
      // the hand-over sub-lists (the fixed scratch has no room for them):
      // sub-list q takes the batches of rows waves q, q + kDeferLists, ...
      const int64_t waves_q = (rows_grid + kDeferLists - 1) / kDeferLists;
      const int64_t batches_w = (n_batch + rows_grid - 1) / rows_grid;
      const int64_t cap = waves_q * batches_w * 4;
      if (!c->d_dcnt)
        HIP_TRY(c, hipMalloc((void**)&c->d_dcnt, (size_t)kDeferLists * kDeferStride * sizeof(uint32_t)));
      if (cap > c->dcap) {
        dfree(c->d_dlist);
        c->dcap = 0;
        HIP_TRY(c, hipMalloc((void**)&c->d_dlist, (size_t)kDeferLists * (size_t)cap * sizeof(int32_t)));
        c->dcap = cap;
      }
      a.dcnt = c->d_dcnt;
      a.dlist = c->d_dlist;
      a.dcap = (int32_t)c->dcap;
    }
  }
  if (ev) HIP_TRY(c, hipEventRecord(ev[0], s));
  // the walk pass over the leaders' lists: a wave per four requests (about
  // two waves per group at the usual group sizes), so the dispatcher
  // balances long walks (popular groups) against short ones
  if (a.grp.keys)
    HIP_TRY(c, ps_launch_group(a, std::max(64, (n_req / 4 + 63) / 64 * 64), s, ev ? ev[1] : nullptr,
                               c->aux, c->fork_ev, c->join_ev));
  else if (ev)
    HIP_TRY(c, hipEventRecord(ev[1], s));
  if (ev) HIP_TRY(c, hipEventRecord(ev[2], s));
  if (rows) {  // four requests per wave
    HIP_TRY(c, ps_launch_lean_rows(a, rows_grid, s));
    a.defer_only = 1;
  } else if (lean) {
    if (!c->lean_wpc) c->lean_wpc = ps_lean_waves_per_cu(c->n_inst);
    const int resident = c->num_cus * c->lean_wpc;
    ScoreArgs la = a;
    la.batch = ps_score_batch(n_req, resident);
    const int lgrid = std::min((n_req + la.batch - 1) / la.batch, resident);
    HIP_TRY(c, ps_launch_lean(la, lgrid, s));
    a.defer_only = 1;
  }
  if (ev) HIP_TRY(c, hipEventRecord(ev[3], s));
  // Finishing what the lean kernel left, the general kernel runs on at most
  // four waves per resident slot: enough waves to balance uneven work (the
  // popular groups), few enough that an empty pass costs little.  With the
  // rows scorer's hand-over lists it runs on its resident waves, each taking
  // an equal share of them.
  int sgrid = lean ? std::min(grid, c->num_cus * 64) : grid;
  if (a.dlist) {
    if (!c->score_wpc) c->score_wpc = ps_score_waves_per_cu(c->n_inst, c->hits_in_lds, rows);
    sgrid = c->num_cus * c->score_wpc;
    if (!c->hits_in_lds && !ps_score_small(c->n_inst)) sgrid = std::min(sgrid, c->scratch_rows);
  }
  HIP_TRY(c, ps_launch_score(a, c->hits_in_lds, sgrid, probe_all, s, rows));
  if (ev) {
    HIP_TRY(c, hipEventRecord(ev[4], s));
    ++c->n_timed;
  }
  return PS_OK;
}

ps_status ps_score_window_dev(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                              const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                              uint32_t* d_sizes, void* hip_stream) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0 || pool_len < 0) return fail(c, PS_E_INVAL, "negative n_req or pool_len");
  if (n_req == 0) return PS_OK;
  if (!d_reqs || !d_out || (pool_len > 0 && !d_pool))
    return fail(c, PS_E_INVAL, "device buffer is NULL");
  DeviceScope ds(c->device);
  return launch_score(c, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes, nullptr,
                      (hipStream_t)hip_stream);
}

ps_status ps_score_window_dev_fixed(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                                    const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                                    uint32_t* d_sizes, void* hip_stream) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0 || pool_len < 0) return fail(c, PS_E_INVAL, "negative n_req or pool_len");
  if (n_req > kFixedMaxReq)
    return fail(c, PS_E_RANGE, "n_req %d exceeds the fixed scratch's %d requests per call", n_req,
                kFixedMaxReq);
  if (n_req == 0) return PS_OK;
  if (!d_reqs || !d_out || (pool_len > 0 && !d_pool))
    return fail(c, PS_E_INVAL, "device buffer is NULL");
  if (c->device >= kMaxDevices) return fail(c, PS_E_STATE, "no fixed scratch on device %d", c->device);
  DeviceScope ds(c->device);
  hipStream_t s = (hipStream_t)hip_stream;
  unsigned char* base = nullptr;
  uint64_t gen = 0;
  bool wrap = false;
  {
    std::lock_guard<std::mutex> lk(g_fixed_mu);
    FixedScratch& f = g_fixed[c->device];
    base = f.ptr;
    if (++f.gen > kGroupGenMax) {
      f.gen = 1;
      wrap = true;
    }
    gen = f.gen;
  }
  if (!base) return fail(c, PS_E_STATE, "fixed scratch was not set up on device %d", c->device);
  if (wrap) HIP_TRY(c, clear_fixed(base, s));
  if (pool_len >= ((int64_t)1 << kGroupGenShift) - 1)  // too long for tagged keys: no groups
    return launch_score(c, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes, nullptr, s);
  unsigned long long* keys = (unsigned long long*)(base + kFixedOffKeys);
  uint32_t* head = (uint32_t*)(base + kFixedOffHead);
  const GroupTab g{keys,
                   keys + kFixedSlots,
                   (uint2*)(base + kFixedOffRec),
                   (uint32_t*)(base + kFixedOffSlot),
                   (uint32_t*)(base + kFixedOffPop),
                   head,
                   (uint32_t)(kFixedPopBytes / ((size_t)c->n_inst * sizeof(uint32_t))),
                   kFixedSlots - 1u,
                   gen,
                   (unsigned long long*)(base + kFixedOffList),
                   head + kListCtrWords * (1u + kXcds * (uint32_t)(gen & 1u)),
                   head + kListCtrWords * (1u + kXcds * (uint32_t)((gen + 1u) & 1u)),
                   kFixedListCap,
                   (uint32_t)(8 * c->num_cus)};
  return launch_score(c, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes, nullptr, s, &g);
}

ps_status ps_set_timing(ps_ctx* c, int32_t on) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  c->timing = on != 0;
  c->n_timed = 0;
  return PS_OK;
}

// Mean milliseconds between consecutive timing events of the timed calls:
// part k spans events k .. k + 1.  Starts a new count.
static ps_status read_parts(ps_ctx* c, int32_t* n_calls, double* ms) {
  if (c->n_timed == 0) return fail(c, PS_E_STATE, "no timed scoring call to read");
  DeviceScope ds(c->device);
  for (int k = 0; k + 1 < kTimingEvents; ++k) ms[k] = 0.0;
  for (int32_t n = 0; n < c->n_timed; ++n) {
    hipEvent_t* ev = &c->ev[kTimingEvents * (size_t)n];
    HIP_TRY(c, hipEventSynchronize(ev[kTimingEvents - 1]));
    for (int k = 0; k + 1 < kTimingEvents; ++k) {
      float t = 0.0f;
      HIP_TRY(c, hipEventElapsedTime(&t, ev[k], ev[k + 1]));
      ms[k] += t;
    }
  }
  for (int k = 0; k + 1 < kTimingEvents; ++k) ms[k] /= c->n_timed;
  *n_calls = c->n_timed;
  c->n_timed = 0;
  return PS_OK;
}

ps_status ps_read_timing(ps_ctx* c, int32_t* n_calls, float* ms_group, float* ms_score) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!n_calls || !ms_group || !ms_score) return fail(c, PS_E_INVAL, "output is NULL");
  double ms[kTimingEvents - 1];
  ps_status st = read_parts(c, n_calls, ms);
  if (st != PS_OK) return st;
  *ms_group = (float)(ms[0] + ms[1]);
  *ms_score = (float)(ms[2] + ms[3]);
  return PS_OK;
}

ps_status ps_read_kernel_timing(ps_ctx* c, int32_t* n_calls, float* ms) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!n_calls || !ms) return fail(c, PS_E_INVAL, "output is NULL");
  double t[kTimingEvents - 1];
  ps_status st = read_parts(c, n_calls, t);
  if (st != PS_OK) return st;
  for (int k = 0; k + 1 < kTimingEvents; ++k) ms[k] = (float)t[k];
  return PS_OK;
}

ps_status ps_probe_hits_dev(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                            const ps_req* d_reqs, int32_t n_req, uint32_t* d_hits,
                            void* hip_stream) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0 || pool_len < 0) return fail(c, PS_E_INVAL, "negative n_req or pool_len");
  if (n_req == 0) return PS_OK;
  if (!d_reqs || !d_hits || (pool_len > 0 && !d_pool))
    return fail(c, PS_E_INVAL, "device buffer is NULL");
  DeviceScope ds(c->device);
  return launch_score(c, d_pool, pool_len, d_reqs, n_req, nullptr, nullptr, d_hits,
                      (hipStream_t)hip_stream);
}

ps_status ps_score_window(ps_ctx* c, const uint64_t* pool, int64_t pool_len, const ps_req* reqs,
                          int32_t n_req, ps_result* out) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0) return fail(c, PS_E_INVAL, "negative n_req");
  if (n_req == 0) return PS_OK;
  if (!out) return fail(c, PS_E_INVAL, "out is NULL");
  ps_status st = check_reqs_host(c, pool, pool_len, reqs, n_req);
  if (st != PS_OK) return st;
  DeviceScope ds(c->device);
  void *dp, *dr, *dout;
  if ((st = stage_buffer(c, 0, (size_t)pool_len * sizeof(uint64_t), &dp)) != PS_OK) return st;
  if ((st = stage_buffer(c, 1, (size_t)n_req * sizeof(ps_req), &dr)) != PS_OK) return st;
  if ((st = stage_buffer(c, 2, (size_t)n_req * sizeof(ps_result), &dout)) != PS_OK) return st;
  hipStream_t s = c->stream;
  if (pool_len)
    HIP_TRY(c, hipMemcpyAsync(dp, pool, (size_t)pool_len * sizeof(uint64_t), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(dr, reqs, (size_t)n_req * sizeof(ps_req), hipMemcpyHostToDevice, s));
  st = launch_score(c, (const uint64_t*)dp, pool_len, (const ps_req*)dr, n_req, (ps_result*)dout,
                    nullptr, nullptr, s);
  if (st != PS_OK) return st;
  HIP_TRY(c, hipMemcpyAsync(out, dout, (size_t)n_req * sizeof(ps_result), hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  return PS_OK;
}

// After placements were committed on the device (work queued on `s`, the
// dropped-block count in d_counter): read the counters back and rebuild the
// derived data the window kernel reads (sorted rooms, key order, prefix
// index).  Synchronous.
static ps_status after_commit(ps_ctx* c, hipStream_t s, int64_t* n_dropped) {
  unsigned long long dropped = 0;
  HIP_TRY(c, hipMemcpyAsync(&dropped, c->d_counter, sizeof dropped, hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipMemcpyAsync(c->h_state.data(), c->d_inst, c->h_state.size() * sizeof(InstState),
                            hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipMemcpyAsync(c->h_count.data(), c->t.count, c->h_count.size() * sizeof(uint32_t),
                            hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  std::vector<int64_t> rs = rooms_of(c->h_state, c->h_model);
  const std::vector<TopRoom> tr = top_rooms(rs);
  HIP_TRY(c, hipMemcpy(c->d_rtop, tr.data(), tr.size() * sizeof(TopRoom), hipMemcpyHostToDevice));
  std::sort(rs.begin(), rs.end());
  HIP_TRY(c, hipMemcpy(c->d_room_sorted, rs.data(), rs.size() * sizeof(int64_t), hipMemcpyHostToDevice));
  const std::vector<uint32_t> o0 = key_order(c->h_state);
  HIP_TRY(c, hipMemcpy(c->d_order0, o0.data(), o0.size() * sizeof(uint32_t), hipMemcpyHostToDevice));
  const std::vector<InstState> ik = states_in_order(c->h_state, o0);
  HIP_TRY(c, hipMemcpy(c->d_inst_key, ik.data(), ik.size() * sizeof(InstState), hipMemcpyHostToDevice));
  HIP_TRY(c, ps_build_index(c->t, c->n_inst, c->h_count.data(), &c->x, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  const ps_status lst = refresh_lmax(c);
  if (lst != PS_OK) return lst;
  if (n_dropped) *n_dropped = (int64_t)dropped;
  return PS_OK;
}

ps_status ps_commit(ps_ctx* c, const uint64_t* pool, int64_t pool_len, const ps_req* reqs,
                    const int32_t* inst, int32_t n, int64_t* n_dropped) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n < 0) return fail(c, PS_E_INVAL, "negative n");
  if (n_dropped) *n_dropped = 0;
  if (n == 0) return PS_OK;
  if (!inst) return fail(c, PS_E_INVAL, "inst is NULL");
  ps_status st = check_reqs_host(c, pool, pool_len, reqs, n);
  if (st != PS_OK) return st;
  const int32_t ni = c->n_inst;
  const int64_t bs = c->h_model.bs;
  std::vector<int32_t> cnt((size_t)ni, 0);
  std::vector<int64_t> add((size_t)ni, 0);
  for (int32_t k = 0; k < n; ++k) {
    const int32_t i = inst[k];
    if (i < -1 || i >= ni) return fail(c, PS_E_RANGE, "entry %d: instance %d outside [-1, %d)", k, i, ni);
    if (i < 0) continue;
    cnt[(size_t)i] += 1;
    add[(size_t)i] += ((int64_t)reqs[k].pre_len + reqs[k].tail_len) * bs;
  }
  std::vector<int32_t> grp_off, grp_inst;
  for (int32_t i = 0; i < ni; ++i) {
    const InstState& s = c->h_state[(size_t)i];
    if (!cnt[(size_t)i]) continue;
    if (s.Q + cnt[(size_t)i] > PS_MAX_DQ)
      return fail(c, PS_E_RANGE, "instance %d: queued would exceed %d", i, PS_MAX_DQ);
    if (s.P + add[(size_t)i] > PS_MAX_PENDING || s.S + add[(size_t)i] > PS_MAX_CONTEXT)
      return fail(c, PS_E_RANGE, "instance %d: token counters would exceed their limits", i);
  }
  // entries grouped by instance, array order kept inside a group
  std::vector<int32_t> start((size_t)ni + 1, 0);
  for (int32_t i = 0; i < ni; ++i) start[(size_t)i + 1] = start[(size_t)i] + cnt[(size_t)i];
  std::vector<int32_t> order((size_t)start[(size_t)ni]);
  {
    std::vector<int32_t> fill(start.begin(), start.end() - 1);
    for (int32_t k = 0; k < n; ++k)
      if (inst[k] >= 0) order[(size_t)fill[(size_t)inst[k]]++] = k;
  }
  for (int32_t i = 0; i < ni; ++i)
    if (cnt[(size_t)i]) {
      grp_inst.push_back(i);
      grp_off.push_back(start[(size_t)i]);
    }
  grp_off.push_back((int32_t)order.size());
  if (grp_inst.empty()) return PS_OK;

  DeviceScope ds(c->device);
  void *dp, *dr, *dx;
  const size_t n_grp = grp_inst.size();
  const size_t aux = (order.size() + 2 * n_grp + 1) * sizeof(int32_t);
  if ((st = stage_buffer(c, 0, (size_t)pool_len * sizeof(uint64_t), &dp)) != PS_OK) return st;
  if ((st = stage_buffer(c, 1, (size_t)n * sizeof(ps_req), &dr)) != PS_OK) return st;
  if ((st = stage_buffer(c, 2, aux, &dx)) != PS_OK) return st;
  int32_t* d_order = (int32_t*)dx;
  int32_t* d_grp_off = d_order + order.size();
  int32_t* d_grp_inst = d_grp_off + n_grp + 1;
  hipStream_t s = c->stream;
  HIP_TRY(c, hipMemcpyAsync(dp, pool, (size_t)pool_len * sizeof(uint64_t), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(dr, reqs, (size_t)n * sizeof(ps_req), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(d_order, order.data(), order.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(d_grp_off, grp_off.data(), grp_off.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(d_grp_inst, grp_inst.data(), n_grp * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemsetAsync(c->d_counter, 0, sizeof(unsigned long long), s));
  CommitArgs ca{c->t, c->d_inst, c->d_room, c->d_model, (const uint64_t*)dp, (const ps_req*)dr,
                d_order, d_grp_off, d_grp_inst, (int32_t)n_grp, (uint32_t)c->cap, c->d_counter};
  HIP_TRY(c, ps_launch_commit(ca, s));
  return after_commit(c, s, n_dropped);
}

static bool req_ok_host(const ps_req& q, int64_t pool_len) {
  return q.pre_len >= 0 && q.tail_len >= 0 && q.pre_off >= 0 && q.tail_off >= 0 &&
         q.pre_off <= pool_len && q.tail_off <= pool_len && q.pre_len <= pool_len - q.pre_off &&
         q.tail_len <= pool_len - q.tail_off && (int64_t)q.pre_len + q.tail_len <= PS_MAX_CHAIN;
}

// Shared body of the per-arrival scheduler and the replay: launches of the
// hits pass and the single-workgroup scheduler over chunks of requests,
// then the refresh of the derived data.
static ps_status run_sequential(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                                const ps_req* d_reqs, int32_t n_req, const int32_t* d_forced,
                                ps_result* d_out, uint32_t* d_sizes, int64_t* n_dropped,
                                hipStream_t s) {
  const int32_t ni = c->n_inst;
  const size_t per_req = (size_t)ni * sizeof(uint32_t);
  const int32_t chunk = (int32_t)std::max<size_t>(1, std::min<size_t>((size_t)n_req, c->seq_budget / per_req));
  const size_t need = (size_t)chunk * (size_t)ni;
  if (need > c->seq_hits_cap) {
    dfree(c->d_seq_hits);
    c->seq_hits_cap = 0;
    HIP_TRY(c, hipMalloc(&c->d_seq_hits, need * sizeof(uint32_t)));
    c->seq_hits_cap = need;
  }
  HIP_TRY(c, hipMemsetAsync(c->d_counter, 0, sizeof(unsigned long long), s));
  const int threads = kSeqMaxThreads;  // every step of a request uses the whole workgroup
  // Speculative batches: Algorithm 1 with a keyed selector (the Random and
  // H-C-Q choices are not a least key, so they are always scored in full)
  const uint32_t sel = c->h_model.sel;
  const bool spec = !d_forced && c->spec_batch > 0 && sel != PS_SEL_RANDOM && sel != PS_SEL_HCQ;
  int32_t step = chunk;
  if (spec) {
    step = std::min(chunk, c->spec_batch);
    if (c->spec_cap < step) {
      dfree(c->d_spec);
      c->spec_cap = 0;
      HIP_TRY(c, hipMalloc(&c->d_spec, (size_t)step * sizeof(SpecRec)));
      c->spec_cap = step;
    }
  }
  if (!c->d_seq_stats) HIP_TRY(c, hipMalloc(&c->d_seq_stats, 2 * sizeof(unsigned long long)));
  HIP_TRY(c, hipMemsetAsync(c->d_seq_stats, 0, 2 * sizeof(unsigned long long), s));
  for (int32_t r0 = 0; r0 < n_req; r0 += step) {
    const int32_t r1 = std::min(n_req, r0 + step);
    ScoreArgs pa{};
    pa.t = c->t;
    pa.x = c->x;
    pa.inst = c->d_inst;
    pa.room = c->d_room;
    pa.model = c->d_model;
    pa.pool = d_pool;
    pa.pool_len = pool_len;
    pa.reqs = d_reqs + r0;
    pa.n_req = r1 - r0;
    pa.n_inst = ni;
    pa.hits_out = c->d_seq_hits;
    const int grid = std::min(r1 - r0, std::max(1, c->num_cus) * 32);
    HIP_TRY(c, ps_launch_score(pa, c->hits_in_lds, grid, true, s));
    SeqArgs q{c->t, c->d_inst, c->d_room, c->d_model, d_pool, pool_len, d_reqs, r0, r1, ni,
              c->d_seq_hits, d_forced, d_out, d_sizes, (uint32_t)c->cap, c->d_counter,
              nullptr, c->d_seq_stats};
    if (spec) {
      HIP_TRY(c, ps_launch_spec(q, c->d_spec, s));
      q.spec = c->d_spec;
    }
    HIP_TRY(c, ps_launch_seq(q, threads, s));
  }
  return after_commit(c, s, n_dropped);
}

ps_status ps_set_schedule_budget(ps_ctx* c, int64_t bytes) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (bytes < 0) return fail(c, PS_E_INVAL, "negative budget");
  c->seq_budget = bytes == 0 ? ((size_t)256 << 20) : (size_t)bytes;
  return PS_OK;
}

ps_status ps_set_schedule_speculation(ps_ctx* c, int32_t batch) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (batch < 0 || batch > kSpecBatch)
    return fail(c, PS_E_INVAL, "speculative batch %d outside [0, %d]", batch, kSpecBatch);
  c->spec_batch = batch;
  return PS_OK;
}

ps_status ps_read_schedule_stats(ps_ctx* c, int64_t* n_spec, int64_t* n_full) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  unsigned long long v[2] = {0, 0};
  if (c->d_seq_stats) {
    DeviceScope ds(c->device);
    HIP_TRY(c, hipMemcpy(v, c->d_seq_stats, sizeof v, hipMemcpyDeviceToHost));
  }
  if (n_spec) *n_spec = (int64_t)v[0];
  if (n_full) *n_full = (int64_t)v[1];
  return PS_OK;
}

ps_status ps_schedule_window_dev(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                                 const ps_req* d_reqs, int32_t n_req, ps_result* d_out,
                                 uint32_t* d_sizes, int64_t* n_dropped, void* hip_stream) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0 || pool_len < 0) return fail(c, PS_E_INVAL, "negative n_req or pool_len");
  if (n_dropped) *n_dropped = 0;
  if (n_req == 0) return PS_OK;
  if (!d_reqs || !d_out || (pool_len > 0 && !d_pool))
    return fail(c, PS_E_INVAL, "device buffer is NULL");
  // Every placement needs A + 1 <= B_max and S + L <= M_KV, which bounds the
  // counters an instance can reach; they must stay inside their limits.
  const DevModel& m = c->h_model;
  for (int32_t i = 0; i < c->n_inst; ++i) {
    const InstState& st = c->h_state[(size_t)i];
    if ((int64_t)m.b_max - 1 - st.D > PS_MAX_DQ)
      return fail(c, PS_E_RANGE, "instance %d: B_max - 1 - D exceeds the queued limit %d", i, PS_MAX_DQ);
    const int64_t grow = std::max<int64_t>(0, m.kv_cap - st.S);
    if (st.P + grow > PS_MAX_PENDING || st.S + grow > PS_MAX_CONTEXT)
      return fail(c, PS_E_RANGE, "instance %d: M_KV allows token counters beyond their limits", i);
  }
  DeviceScope ds(c->device);
  return run_sequential(c, d_pool, pool_len, d_reqs, n_req, nullptr, d_out, d_sizes, n_dropped,
                        (hipStream_t)hip_stream);
}

ps_status ps_replay_window_dev(ps_ctx* c, const uint64_t* d_pool, int64_t pool_len,
                               const ps_req* d_reqs, int32_t n_req, const int32_t* d_inst,
                               ps_result* d_out, int64_t* n_dropped, void* hip_stream) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n_req < 0 || pool_len < 0) return fail(c, PS_E_INVAL, "negative n_req or pool_len");
  if (n_dropped) *n_dropped = 0;
  if (n_req == 0) return PS_OK;
  if (!d_reqs || !d_out || !d_inst || (pool_len > 0 && !d_pool))
    return fail(c, PS_E_INVAL, "device buffer is NULL");
  DeviceScope ds(c->device);
  hipStream_t s = (hipStream_t)hip_stream;
  std::vector<int32_t> inst((size_t)n_req);
  std::vector<ps_req> reqs((size_t)n_req);
  HIP_TRY(c, hipMemcpyAsync(inst.data(), d_inst, inst.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipMemcpyAsync(reqs.data(), d_reqs, reqs.size() * sizeof(ps_req), hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  const int32_t ni = c->n_inst;
  const int64_t bs = c->h_model.bs;
  std::vector<int32_t> cnt((size_t)ni, 0);
  std::vector<int64_t> add((size_t)ni, 0);
  for (int32_t k = 0; k < n_req; ++k) {
    const int32_t i = inst[(size_t)k];
    if (i < -1 || i >= ni) return fail(c, PS_E_RANGE, "entry %d: instance %d outside [-1, %d)", k, i, ni);
    if (i < 0 || !req_ok_host(reqs[(size_t)k], pool_len)) continue;
    cnt[(size_t)i] += 1;
    add[(size_t)i] += ((int64_t)reqs[(size_t)k].pre_len + reqs[(size_t)k].tail_len) * bs;
  }
  for (int32_t i = 0; i < ni; ++i) {
    const InstState& st = c->h_state[(size_t)i];
    if (st.Q + cnt[(size_t)i] > PS_MAX_DQ)
      return fail(c, PS_E_RANGE, "instance %d: queued would exceed %d", i, PS_MAX_DQ);
    if (st.P + add[(size_t)i] > PS_MAX_PENDING || st.S + add[(size_t)i] > PS_MAX_CONTEXT)
      return fail(c, PS_E_RANGE, "instance %d: token counters would exceed their limits", i);
  }
  return run_sequential(c, d_pool, pool_len, d_reqs, n_req, d_inst, d_out, nullptr, n_dropped, s);
}

ps_status ps_apply_events(ps_ctx* c, const ps_event* ev, int32_t n) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n < 0 || (n > 0 && !ev)) return fail(c, PS_E_INVAL, "bad event array");
  std::vector<InstState> st = c->h_state;
  for (int32_t k = 0; k < n; ++k) {
    const ps_event& e = ev[k];
    if (e.instance < 0 || e.instance >= c->n_inst)
      return fail(c, PS_E_INVAL, "event %d: instance %d outside [0, %d)", k, e.instance, c->n_inst);
    if (e.tokens < 0) return fail(c, PS_E_INVAL, "event %d: negative tokens", k);
    InstState& s = st[(size_t)e.instance];
    switch (e.kind) {
      case PS_EV_PREFILL_DONE:
        s.Q -= 1;
        s.D += 1;
        s.P -= e.tokens;
        break;
      case PS_EV_DECODE_TOKENS:
        s.S += e.tokens;
        break;
      case PS_EV_FINISHED:
        s.D -= 1;
        s.S -= e.tokens;
        break;
      default:
        return fail(c, PS_E_INVAL, "event %d: unknown kind %d", k, e.kind);
    }
    if (s.D < 0 || s.D > PS_MAX_DQ || s.Q < 0 || s.Q > PS_MAX_DQ || s.P < 0 ||
        s.P > PS_MAX_PENDING || s.S < 0 || s.S > PS_MAX_CONTEXT)
      return fail(c, PS_E_RANGE, "event %d leaves instance %d outside the counter limits", k,
                  e.instance);
  }
  DeviceScope ds(c->device);
  std::vector<InstState> old = c->h_state;
  c->h_state = st;
  ps_status rc = refresh_derived(c);
  if (rc != PS_OK) c->h_state = old;
  return rc;
}

ps_status ps_feedback_decode(ps_ctx* c, const int32_t* batch, const int64_t* ctx_tok,
                             const float* measured_s, int32_t n) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n < 0 || (n > 0 && (!batch || !ctx_tok || !measured_s)))
    return fail(c, PS_E_INVAL, "bad sample arrays");
  for (int32_t k = 0; k < n; ++k)
    if (batch[k] < 1 || ctx_tok[k] < 0 || !std::isfinite(measured_s[k]) || !(measured_s[k] > 0.0f))
      return fail(c, PS_E_INVAL, "sample %d: batch >= 1, context >= 0, finite positive duration", k);
  std::vector<double> g = c->gamma64;
  const DevModel& m = c->h_model;
  for (int32_t k = 0; k < n; ++k) {
    const int32_t s = segment_of_dev(m, batch[k]);
    const double pred = (double)m.seg[s][0] + (double)m.seg[s][1] * (double)batch[k] +
                        (double)m.seg[s][2] * (double)ctx_tok[k];
    if (!(pred > 0.0)) continue;
    const double ratio = std::min(2.0, std::max(0.5, (double)measured_s[k] / pred));
    g[(size_t)s] = std::min(2.0, std::max(1.0, 0.98 * g[(size_t)s] + 0.02 * ratio));
  }
  DeviceScope ds(c->device);
  const DevModel keep = c->h_model;
  for (int32_t s = 0; s < m.n_seg; ++s) c->h_model.seg[s][3] = (float)g[(size_t)s];
  const ps_status rc = upload_model(c);
  if (rc != PS_OK) {
    c->h_model = keep;
    return rc;
  }
  c->gamma64 = g;
  return PS_OK;
}

ps_status ps_feedback_output(ps_ctx* c, const int32_t* out_len, int32_t n) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (n < 0 || (n > 0 && !out_len)) return fail(c, PS_E_INVAL, "bad length array");
  for (int32_t k = 0; k < n; ++k)
    if (out_len[k] < 0) return fail(c, PS_E_INVAL, "output length %d is negative", k);
  if (n == 0) return PS_OK;
  std::vector<int32_t> ring = c->lout_ring;
  int64_t seen = c->lout_seen;
  if (ring.size() < (size_t)PS_LOUT_WINDOW) ring.resize(PS_LOUT_WINDOW, 0);
  for (int32_t k = 0; k < n; ++k) ring[(size_t)((seen++) % PS_LOUT_WINDOW)] = out_len[k];
  const size_t mlen = (size_t)std::min<int64_t>(seen, PS_LOUT_WINDOW);
  std::vector<int32_t> win(ring.begin(), ring.begin() + (long)mlen);
  std::nth_element(win.begin(), win.begin() + (long)((mlen - 1) / 2), win.end());
  const float lout = (float)win[(mlen - 1) / 2];
  DeviceScope ds(c->device);
  const DevModel keep = c->h_model;
  c->h_model.lout1 = std::max(1.0f, lout);
  const ps_status rc = upload_model(c);
  if (rc != PS_OK) {
    c->h_model = keep;
    return rc;
  }
  c->lout_ring = ring;
  c->lout_seen = seen;
  c->lout_raw = lout;
  return PS_OK;
}

ps_status ps_read_model(ps_ctx* c, float* gamma, float* lout, int32_t* n_seg) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (gamma)
    for (int32_t s = 0; s < c->h_model.n_seg; ++s) gamma[s] = c->h_model.seg[s][3];
  if (lout) *lout = c->lout_raw;
  if (n_seg) *n_seg = c->h_model.n_seg;
  return PS_OK;
}

ps_status ps_read_state(ps_ctx* c, int32_t* decoding, int32_t* queued, int64_t* pending_tok,
                        int64_t* ctx_tok, int64_t* cached_blocks) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  for (int32_t i = 0; i < c->n_inst; ++i) {
    const InstState& s = c->h_state[(size_t)i];
    if (decoding) decoding[i] = s.D;
    if (queued) queued[i] = s.Q;
    if (pending_tok) pending_tok[i] = s.P;
    if (ctx_tok) ctx_tok[i] = s.S;
    if (cached_blocks) cached_blocks[i] = c->h_count[(size_t)i];
  }
  return PS_OK;
}

ps_status ps_table_info(ps_ctx* c, int64_t* slots_per_table, int64_t* table_bytes,
                        int32_t* hits_in_lds) {
  if (!c) return fail(nullptr, PS_E_INVAL, "ctx is NULL");
  if (!c->loaded) return fail(c, PS_E_STATE, "ps_load_instances has not succeeded yet");
  if (slots_per_table) *slots_per_table = c->t.slots;
  if (table_bytes) *table_bytes = c->t.slots * (int64_t)c->n_inst * (int64_t)sizeof(uint64_t);
  if (hits_in_lds) *hits_in_lds = c->hits_in_lds ? 1 : 0;
  return PS_OK;
}

}  // extern "C"
