// Edge ordering for the segmented reduction: a stable LSD radix sort of the
// destination (or source) index with 8-bit digits, the segment offsets by
// binary search over the sorted keys, and device-side input validation.
//
// Stability: every pass is a stable counting sort; within a block the items
// are ranked in their original order (wave ballots give the rank among equal
// digits inside a wave, waves are ordered by index, tiles by block), so equal
// keys keep the original edge order and perm/offsets are exact integers.
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

constexpr int kSortThreads = 256;
constexpr int kItemsPerThread = 4;  // 1024 keys per block: more blocks in flight (16 measured slower)
constexpr int kSortTile = kSortThreads * kItemsPerThread;
constexpr int kDigits = 256;

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

__global__ __launch_bounds__(kSortThreads) void k_digit_hist(const int32_t* __restrict__ keys, int E, int shift,
                                                            int n_blocks, int32_t* __restrict__ hist) {
  __shared__ int32_t h[kDigits];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * kSortTile;
  for (int i = 0; i < kItemsPerThread; ++i) {
    const int idx = base + i * kSortThreads + threadIdx.x;
    if (idx < E) atomicAdd(&h[(keys[idx] >> shift) & (kDigits - 1)], 1);
  }
  __syncthreads();
  hist[threadIdx.x * n_blocks + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan of n ints in place, one block of 1024 threads.
__global__ __launch_bounds__(1024) void k_scan_exclusive(int32_t* __restrict__ a, int n) {
  __shared__ int32_t part[1024];
  const int per = (n + 1023) / 1024;
  const int lo = min(n, int(threadIdx.x) * per), hi = min(n, lo + per);
  int32_t s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t t = threadIdx.x >= unsigned(off) ? part[threadIdx.x - off] : 0;
    __syncthreads();
    part[threadIdx.x] += t;
    __syncthreads();
  }
  int32_t run = part[threadIdx.x] - s;
  for (int i = lo; i < hi; ++i) {
    const int32_t v = a[i];
    a[i] = run;
    run += v;
  }
}

// Exclusive scan of each digit's row hist[digit][0 .. n_blocks) in place,
// one wave (block) per digit, and the row's total into totals[digit].
__global__ __launch_bounds__(kWave) void k_scan_rows(int32_t* __restrict__ hist, int n_blocks,
                                                     int32_t* __restrict__ totals) {
  const int lane = threadIdx.x;
  int32_t* row = hist + size_t(blockIdx.x) * n_blocks;
  int32_t carry = 0;
  for (int b0 = 0; b0 < n_blocks; b0 += kWave) {
    const int b = b0 + lane;
    const int32_t v = b < n_blocks ? row[b] : 0;
    int32_t x = v;  // inclusive scan over the wave
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (b < n_blocks) row[b] = carry + x - v;
    carry += __shfl(x, kWave - 1);
  }
  if (lane == 0) totals[blockIdx.x] = carry;
}

// The scatter of one pass: each block's items go to base[digit] (the
// exclusive scan of the digit totals, formed here) + the row-scanned count of
// earlier blocks + the rank within the block.
__global__ __launch_bounds__(kSortThreads) void k_digit_scatter(const int32_t* __restrict__ keys_in,
                                                               const int32_t* __restrict__ vals_in, int E,
                                                               int shift, int n_blocks,
                                                               const int32_t* __restrict__ hist,
                                                               const int32_t* __restrict__ totals,
                                                               int32_t* __restrict__ keys_out,
                                                               int32_t* __restrict__ vals_out) {
  constexpr int kWaves = kSortThreads / kWave;
  static_assert(kSortThreads == kDigits, "one thread per digit");
  __shared__ int32_t run[kDigits];
  __shared__ int32_t wcnt[kWaves][kDigits];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  {
    // exclusive scan of the digit totals: per wave, then the wave sums
    const int32_t v = totals[tid];
    int32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == kWave - 1) wcnt[0][wave] = x;
    __syncthreads();
    int32_t base = x - v;
    for (int w = 0; w < wave; ++w) base += wcnt[0][w];
    run[tid] = base + hist[tid * n_blocks + blockIdx.x];
    __syncthreads();
  }
  for (int w = 0; w < kWaves; ++w) wcnt[w][tid] = 0;
  __syncthreads();
  const uint64_t lt_mask = lane == 0 ? 0ull : (~0ull >> (kWave - lane));
  const int base = blockIdx.x * kSortTile;
  for (int it = 0; it < kItemsPerThread; ++it) {
    const int idx = base + it * kSortThreads + tid;
    const bool valid = idx < E;
    const int32_t key = valid ? keys_in[idx] : 0;
    const int32_t val = valid ? (vals_in ? vals_in[idx] : idx) : 0;
    const int digit = (key >> shift) & (kDigits - 1);
    uint64_t peers = __ballot(valid);
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (digit >> bit) & 1;
      const uint64_t b = __ballot(on);
      peers &= on ? b : ~b;
    }
    const int rank = __popcll(peers & lt_mask);
    if (valid && rank == 0) wcnt[wave][digit] = __popcll(peers);
    __syncthreads();
    if (valid) {
      int pos = run[digit] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][digit];
      keys_out[pos] = key;
      vals_out[pos] = val;
    }
    __syncthreads();
    int32_t add = 0;
    for (int w = 0; w < kWaves; ++w) {
      add += wcnt[w][tid];
      wcnt[w][tid] = 0;
    }
    run[tid] += add;
    __syncthreads();
  }
}

// offsets[k] = first index i with sorted_keys[i] >= k (E if none), for k in
// [0, n_keys]: one wave per key, a 64-way search.  Each round the 64 lanes
// compare the keys at 64 positions spread over the remaining range and the
// count of keys below k (a ballot) narrows it 65-fold, so 151 k edges take
// three dependent loads instead of the 17 of a binary search; once at most
// 64 positions remain, one load per lane settles it.  For keys that are not
// sorted the result is still some index in [0, E].
__device__ __forceinline__ void wave_lower_bound(const int32_t* __restrict__ sorted_keys, int E, int k, int lane,
                                                 int32_t* __restrict__ out) {
  int lo = 0, hi = E;  // the answer lies in [lo, hi]
  while (hi - lo > kWave) {
    const int q = lo + int(int64_t(hi - lo) * (lane + 1) / (kWave + 1));  // lo <= q < hi
    const unsigned long long below = __ballot(sorted_keys[q] < k);
    const int c = __popcll(below);
    const int q_lo = lo + int(int64_t(hi - lo) * c / (kWave + 1));  // probe c - 1 (c > 0)
    const int q_hi = lo + int(int64_t(hi - lo) * (c + 1) / (kWave + 1));  // probe c (c < 64)
    const int nlo = c > 0 ? q_lo + 1 : lo;
    const int nhi = c < kWave ? q_hi : hi;
    lo = nlo;
    hi = nhi;
  }
  const bool below = lo + lane < hi && sorted_keys[lo + lane] < k;
  const int c = __popcll(__ballot(below));
  if (lane == 0) *out = lo + c;
}

__global__ void k_offsets(const int32_t* __restrict__ sorted_keys, int E, int n_keys, int32_t* __restrict__ offsets) {
  const int k = int((size_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave);
  if (k > n_keys) return;  // whole waves
  wave_lower_bound(sorted_keys, E, k, threadIdx.x % kWave, offsets + k);
}

// Pre-sorted keys in one launch: perm[i] = i for every i < E (grid-stride),
// and the offsets as in k_offsets, one wave per key.
__global__ void k_iota_offsets(const int32_t* __restrict__ sorted_keys, int E, int n_keys, int32_t* __restrict__ perm,
                               int32_t* __restrict__ offsets) {
  const size_t gid = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (size_t i = gid; i < size_t(E); i += size_t(gridDim.x) * blockDim.x) perm[i] = int32_t(i);
  const int k = int(gid / kWave);
  if (k > n_keys) return;
  wave_lower_bound(sorted_keys, E, k, threadIdx.x % kWave, offsets + k);
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, size_t n) {
  const size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

__global__ void k_validate(int N, int E, const int32_t* __restrict__ ei, const float* __restrict__ vec,
                           int check_sorted, int32_t* __restrict__ flags) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E) return;
  const int s = ei[i], t = ei[E + i];
  if (s < 0 || s >= N || t < 0 || t >= N) atomicOr(&flags[0], 1);
  if (check_sorted && i + 1 < E && t > ei[E + i + 1]) atomicOr(&flags[1], 1);
  const float x = vec[3 * i], y = vec[3 * i + 1], z = vec[3 * i + 2];
  const float n2 = x * x + y * y + z * z;
  if (!(n2 > 0.f) || !isfinite(n2)) atomicOr(&flags[2], 1);
}

}  // namespace

SortPlan sort_plan(int n_keys, int E) {
  SortPlan p{};
  p.n_keys = n_keys;
  p.E = E;
  int bits = 0;
  while (bits < 31 && (int64_t(1) << bits) < int64_t(n_keys)) ++bits;
  p.passes = (bits + 7) / 8;
  p.n_blocks = (E + kSortTile - 1) / kSortTile;
  const size_t e4 = align256(size_t(E) * 4);
  p.bytes = 4 * e4 + align256(size_t(kDigits) * p.n_blocks * 4) + align256(size_t(kDigits) * 4);
  return p;
}

hipError_t launch_scan_exclusive(int32_t* a, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_scan_exclusive<<<dim3(1), dim3(1024), 0, s>>>(a, n);
  return hipGetLastError();
}

hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  k_fill_u32<<<dim3(unsigned((n + 255) / 256)), dim3(256), 0, s>>>(static_cast<uint32_t*>(ptr), n);
  return hipGetLastError();
}

hipError_t launch_offsets_presorted(int n_keys, int E, const int32_t* sorted_keys, int32_t* perm, int32_t* offsets,
                                    hipStream_t s) {
  // one wave per key (n_keys + 1 of them); the perm writes stride over the grid
  const size_t threads = size_t(n_keys + 1) * kWave;
  k_iota_offsets<<<dim3(unsigned((threads + 255) / 256)), dim3(256), 0, s>>>(sorted_keys, E, n_keys, perm, offsets);
  return hipGetLastError();
}

hipError_t launch_sort(const SortPlan& plan, const int32_t* keys, int /*key_stride*/, int32_t* perm, int32_t* offsets,
                       void* ws, hipStream_t s) {
  const int E = plan.E;
  if (E == 0 || plan.passes == 0) {
    // no key bits: the stable order is the original order; offsets from the keys themselves
    return launch_offsets_presorted(plan.n_keys, E, keys, perm, offsets, s);
  }
  char* w = static_cast<char*>(ws);
  const size_t e4 = align256(size_t(E) * 4);
  int32_t* kbuf[2] = {reinterpret_cast<int32_t*>(w), reinterpret_cast<int32_t*>(w + e4)};
  int32_t* vbuf[2] = {reinterpret_cast<int32_t*>(w + 2 * e4), reinterpret_cast<int32_t*>(w + 3 * e4)};
  int32_t* hist = reinterpret_cast<int32_t*>(w + 4 * e4);
  int32_t* totals = reinterpret_cast<int32_t*>(w + 4 * e4 + align256(size_t(kDigits) * plan.n_blocks * 4));
  const int nb = plan.n_blocks;
  const int32_t* kin = keys;
  const int32_t* vin = nullptr;
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int shift = 8 * pass;
    int32_t* kout = kbuf[pass & 1];
    int32_t* vout = pass + 1 == plan.passes ? perm : vbuf[pass & 1];
    k_digit_hist<<<dim3(nb), dim3(kSortThreads), 0, s>>>(kin, E, shift, nb, hist);
    k_scan_rows<<<dim3(kDigits), dim3(kWave), 0, s>>>(hist, nb, totals);
    k_digit_scatter<<<dim3(nb), dim3(kSortThreads), 0, s>>>(kin, vin, E, shift, nb, hist, totals, kout, vout);
    kin = kout;
    vin = vout;
  }
  k_offsets<<<dim3(unsigned((size_t(plan.n_keys + 1) * kWave + 255) / 256)), dim3(256), 0, s>>>(kin, E, plan.n_keys,
                                                                                                offsets);
  return hipGetLastError();
}

hipError_t launch_validate(int N, int E, const int32_t* edge_index, const float* edge_vec, int check_sorted,
                           int32_t* flags, hipStream_t s) {
  hipError_t e = launch_zero(flags, 4 * sizeof(int32_t), s);
  if (e != hipSuccess) return e;
  if (E > 0)
    k_validate<<<dim3((E + 255) / 256), dim3(256), 0, s>>>(N, E, edge_index, edge_vec, check_sorted, flags);
  return hipGetLastError();
}

}  // namespace tdn
