// Prefix index build: all (block hash, instance) pairs of the per-instance
// tables, sorted by hash with hipCUB's radix sort (stable, so each hash's
// holders stay in ascending instance order), run-length encoded into one
// entry per distinct hash and inserted into an open-addressing table of
// 16-byte entries.  Runs at ps_load_instances and after ps_commit; not on
// the timed path.

#include <hipcub/hipcub.hpp>

#include <vector>

#include "ps_device.h"

using namespace ps;

namespace {

// Pairs of instance i go to [base[i], base[i] + count[i]) (any order inside
// the range).  A wave whose slots all belong to one instance claims its
// positions with one atomic.
__global__ void extract_kernel(Tables t, int32_t n_inst, const int64_t* base, uint64_t* pk,
                               uint16_t* pv, unsigned int* cursor) {
  const int64_t total = (int64_t)n_inst * t.slots;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int lane = threadIdx.x & 63;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += stride) {
    const uint64_t key = t.keys[k];
    const int32_t i = (int32_t)(k / t.slots);
    const uint64_t act = __ballot(1);
    const int leader = __builtin_ctzll(act);
    const int32_t i0 = __shfl(i, leader);
    int64_t at = -1;
    if (__ballot(i == i0) == act) {
      const uint64_t wm = __ballot(key != 0);
      uint32_t b0 = 0;
      if (lane == leader && wm) b0 = atomicAdd(&cursor[i0], (unsigned int)__popcll(wm));
      b0 = (uint32_t)__shfl((int)b0, leader);
      if (key != 0) at = base[i0] + b0 + __popcll(wm & lt_mask);
    } else if (key != 0) {
      at = base[i] + atomicAdd(&cursor[i], 1u);
    }
    if (at >= 0) {
      pk[at] = key;
      pv[at] = (uint16_t)i;
    }
  }
}

// Popular hashes: set the bits of their holders in their bitmap
// (bitmap number = exclusive scan of the popular flags).
__global__ void bitmap_kernel(GIndex x, const uint32_t* uc, const uint32_t* uo,
                              const uint32_t* pop_rank, const int* n_runs) {
  const int n = *n_runs;
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) {
    if (uc[k] <= kPopular) continue;
    uint64_t* bm = x.bitmaps + (size_t)pop_rank[k] * x.nw;
    for (uint32_t t = 0; t < uc[k]; ++t) {
      const uint32_t id = x.holders[uo[k] + t];
      atomicOr(reinterpret_cast<unsigned long long*>(&bm[id >> 6]), 1ull << (id & 63));
    }
  }
}

__global__ void popular_flag_kernel(const uint32_t* uc, uint32_t* flag, const int* n_runs) {
  const int n = *n_runs;
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x)
    flag[k] = uc[k] > kPopular ? 1u : 0u;
}

__global__ void insert_index_kernel(GIndex x, const uint64_t* uk, const uint32_t* uc,
                                    const uint32_t* uo, const uint32_t* pop_rank,
                                    const int* n_runs, unsigned long long* full) {
  const int n = *n_runs;
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n; k += gridDim.x * blockDim.x) {
    const uint64_t key = uk[k];
    uint32_t b = bucket_of(key, kIndexSalt, x.shift);
    bool done = false;
    for (uint32_t step = 0; step <= x.bmask && !done; ++step) {
      IdxEntry* bp = x.ent + (size_t)b * kSlotsPerBucket;
      for (int s = 0; s < kSlotsPerBucket; ++s) {
        unsigned long long old = atomicCAS(reinterpret_cast<unsigned long long*>(&bp[s].key), 0ull,
                                           (unsigned long long)key);
        if (old == 0ull) {
          bp[s].off = uc[k] > kPopular ? pop_rank[k] : uo[k];
          bp[s].cnt = uc[k];
          done = true;
          break;
        }
      }
      b = (b + 1) & x.bmask;
    }
    if (!done) atomicAdd(full, 1ull);
  }
}

template <class T>
void dfree(T*& p) {
  if (p) (void)hipFree((void*)p);
  p = nullptr;
}

}  // namespace

void ps_free_index(GIndex* x) {
  dfree(x->ent);
  dfree(x->holders);
  dfree(x->bitmaps);
  x->bmask = 0;
  x->shift = 64;
}

#define TRY(call)                   \
  do {                              \
    e = (call);                     \
    if (e != hipSuccess) goto done; \
  } while (0)

hipError_t ps_build_index(const Tables& t, int32_t n_inst, const uint32_t* count_host, GIndex* x,
                          hipStream_t s) {
  hipError_t e = hipSuccess;
  std::vector<int64_t> base((size_t)n_inst + 1, 0);
  for (int32_t i = 0; i < n_inst; ++i) base[(size_t)i + 1] = base[(size_t)i] + count_host[i];
  const int64_t n = base[(size_t)n_inst];
  int64_t* d_base = nullptr;
  unsigned int* d_cursor = nullptr;
  uint64_t *pk = nullptr, *sk = nullptr, *uk = nullptr;
  uint16_t *pv = nullptr, *sv = nullptr;
  uint32_t *uc = nullptr, *uo = nullptr, *pflag = nullptr, *prank = nullptr;
  uint32_t n_pop = 0;
  int* d_runs = nullptr;
  unsigned long long* d_full = nullptr;
  void* tmp = nullptr;
  size_t tmp_bytes = 0, b1 = 0, b2 = 0, b3 = 0;
  int runs = 0;
  unsigned long long full = 0;
  GIndex nx{nullptr, nullptr, nullptr, (uint32_t)((n_inst + 63) / 64), 0, 64};
  const int nn = (int)(n > 0 ? n : 1);
  int64_t buckets = 1;
  int log2b = 0;

  TRY(hipMalloc(&d_base, base.size() * sizeof(int64_t)));
  TRY(hipMalloc(&d_cursor, (size_t)n_inst * sizeof(unsigned int)));
  TRY(hipMalloc(&pk, (size_t)nn * sizeof(uint64_t)));
  TRY(hipMalloc(&sk, (size_t)nn * sizeof(uint64_t)));
  TRY(hipMalloc(&uk, (size_t)nn * sizeof(uint64_t)));
  TRY(hipMalloc(&pv, (size_t)nn * sizeof(uint16_t)));
  TRY(hipMalloc(&sv, (size_t)nn * sizeof(uint16_t)));
  TRY(hipMalloc(&uc, (size_t)nn * sizeof(uint32_t)));
  TRY(hipMalloc(&uo, (size_t)nn * sizeof(uint32_t)));
  TRY(hipMalloc(&pflag, (size_t)nn * sizeof(uint32_t)));
  TRY(hipMalloc(&prank, (size_t)nn * sizeof(uint32_t)));
  TRY(hipMalloc(&d_runs, sizeof(int)));
  TRY(hipMalloc(&d_full, sizeof(unsigned long long)));
  TRY(hipMemcpyAsync(d_base, base.data(), base.size() * sizeof(int64_t), hipMemcpyHostToDevice, s));
  TRY(hipMemsetAsync(d_cursor, 0, (size_t)n_inst * sizeof(unsigned int), s));
  TRY(hipMemsetAsync(d_runs, 0, sizeof(int), s));
  TRY(hipMemsetAsync(d_full, 0, sizeof(unsigned long long), s));
  if (n > 0) {
    const int64_t total = (int64_t)n_inst * t.slots;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(extract_kernel, dim3((unsigned)blocks), dim3(256), 0, s, t, n_inst, d_base,
                       pk, pv, d_cursor);
    TRY(hipGetLastError());
    TRY(hipcub::DeviceRadixSort::SortPairs(nullptr, b1, pk, sk, pv, sv, (int)n, 0, 64, s));
    TRY(hipcub::DeviceRunLengthEncode::Encode(nullptr, b2, sk, uk, uc, d_runs, (int)n, s));
    TRY(hipcub::DeviceScan::ExclusiveSum(nullptr, b3, uc, uo, (int)n, s));
    tmp_bytes = std::max(b1, std::max(b2, b3));
    TRY(hipMalloc(&tmp, tmp_bytes));
    TRY(hipcub::DeviceRadixSort::SortPairs(tmp, tmp_bytes, pk, sk, pv, sv, (int)n, 0, 64, s));
    TRY(hipcub::DeviceRunLengthEncode::Encode(tmp, tmp_bytes, sk, uk, uc, d_runs, (int)n, s));
    TRY(hipMemcpyAsync(&runs, d_runs, sizeof(int), hipMemcpyDeviceToHost, s));
    TRY(hipStreamSynchronize(s));
    TRY(hipcub::DeviceScan::ExclusiveSum(tmp, tmp_bytes, uc, uo, runs, s));
    {
      int blocks = (runs + 255) / 256;
      if (blocks > 65536) blocks = 65536;
      hipLaunchKernelGGL(popular_flag_kernel, dim3(blocks), dim3(256), 0, s, uc, pflag, d_runs);
      TRY(hipGetLastError());
    }
    TRY(hipcub::DeviceScan::ExclusiveSum(tmp, tmp_bytes, pflag, prank, runs, s));
    {
      uint32_t last_flag = 0, last_rank = 0;
      TRY(hipMemcpyAsync(&last_flag, pflag + runs - 1, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
      TRY(hipMemcpyAsync(&last_rank, prank + runs - 1, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
      TRY(hipStreamSynchronize(s));
      n_pop = last_flag + last_rank;
    }
  }
  // table of >= 2 * runs entries in buckets of 8
  while (buckets * kSlotsPerBucket < 2 * (int64_t)runs) {
    buckets <<= 1;
    ++log2b;
  }
  nx.bmask = (uint32_t)(buckets - 1);
  nx.shift = (uint32_t)(64 - log2b);
  TRY(hipMalloc(&nx.ent, (size_t)buckets * kSlotsPerBucket * sizeof(IdxEntry)));
  TRY(hipMemsetAsync(nx.ent, 0, (size_t)buckets * kSlotsPerBucket * sizeof(IdxEntry), s));
  if (n_pop > 0) {
    TRY(hipMalloc(&nx.bitmaps, (size_t)n_pop * nx.nw * sizeof(uint64_t)));
    TRY(hipMemsetAsync(nx.bitmaps, 0, (size_t)n_pop * nx.nw * sizeof(uint64_t), s));
  }
  if (runs > 0) {
    int blocks = (runs + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    nx.holders = sv;  // read by bitmap_kernel
    hipLaunchKernelGGL(insert_index_kernel, dim3(blocks), dim3(256), 0, s, nx, uk, uc, uo, prank,
                       d_runs, d_full);
    TRY(hipGetLastError());
    if (n_pop > 0) {
      hipLaunchKernelGGL(bitmap_kernel, dim3(blocks), dim3(256), 0, s, nx, uc, uo, prank, d_runs);
      TRY(hipGetLastError());
    }
  }
  TRY(hipMemcpyAsync(&full, d_full, sizeof full, hipMemcpyDeviceToHost, s));
  TRY(hipStreamSynchronize(s));
  if (full) {
    e = hipErrorUnknown;
    goto done;
  }
  nx.holders = sv;
  nx.n_pop = n_pop;
  sv = nullptr;
  ps_free_index(x);
  *x = nx;
  nx.ent = nullptr;
  nx.bitmaps = nullptr;
done:
  if (nx.ent) (void)hipFree(nx.ent);
  if (nx.bitmaps) (void)hipFree(nx.bitmaps);
  dfree(d_base);
  dfree(d_cursor);
  dfree(pk);
  dfree(sk);
  dfree(uk);
  dfree(pv);
  dfree(sv);
  dfree(uc);
  dfree(uo);
  dfree(pflag);
  dfree(prank);
  dfree(d_runs);
  dfree(d_full);
  if (tmp) (void)hipFree(tmp);
  return e;
}

hipError_t ps_exclusive_scan_u32(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  size_t bytes = 0;
  hipError_t e = hipcub::DeviceScan::ExclusiveSum(nullptr, bytes, in, out, (int)n, s);
  if (e != hipSuccess) return e;
  void* tmp = nullptr;
  e = hipMalloc(&tmp, bytes);
  if (e != hipSuccess) return e;
  e = hipcub::DeviceScan::ExclusiveSum(tmp, bytes, in, out, (int)n, s);
  hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(tmp);
  return e != hipSuccess ? e : e2;
}
