// Stable LSD radix sort of (uint64 key, int32 value) pairs on gfx950, and the
// device-wide exclusive scan it uses.  8-bit digits, or 9-bit ones where that
// saves a pass (17-18, 25-27 or 33-36 bits to sort, e.g. the 18 brick bits of
// the headline's Morton codes); one pass is
//   k_rs_hist     per-block digit histogram (LDS atomics)   -> hist[digit][block]
//   scan          exclusive scan of hist in digit-major order (global offsets)
//   k_rs_scatter  per-block stable ranking (wave ballots for equal digits,
//                 per-wave digit counts combined in LDS) and scatter.
// The element count is read from device memory, so a sort can be enqueued
// before the host knows how many elements there are.
#include "internal.h"

namespace spc {
namespace {

constexpr int kWave = 64;
constexpr int kItems = 8;                       // elements per thread per block
constexpr int kSortTile = kBlock * kItems;      // 2048 elements per block
constexpr int kMaxDigits = 512;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint64_t lanes_below() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// ---------------------------------------------------------------------------
// Exclusive scan of a uint32 array of `n` elements (three launches, two when
// there are at most kSelfParts chunks).
// ---------------------------------------------------------------------------
constexpr int kScanChunk = 4 * kBlock;          // elements per scan block

template <typename T>
__device__ __forceinline__ T wave_incl(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    T t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T block_excl(T v, T* total) {
  __shared__ T s_w[kBlock / kWave];
  const int wave = threadIdx.x / kWave;
  T inc = wave_incl(v);
  if (lane_id() == kWave - 1) s_w[wave] = inc;
  __syncthreads();
  T base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kBlock / kWave; ++w) {
    if (w < wave) base += s_w[w];
    tot += s_w[w];
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

__global__ __launch_bounds__(kBlock) void k_scan_reduce(const uint32_t* __restrict__ a,
                                                        int64_t n, uint32_t* __restrict__ part) {
  const int64_t base = blockIdx.x * static_cast<int64_t>(kScanChunk) + 4 * threadIdx.x;
  uint32_t v = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u)
    if (base + u < n) v += a[base + u];
  uint32_t tot;
  block_excl<uint32_t>(v, &tot);
  if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_scan_top(uint32_t* __restrict__ part, int64_t np) {
  uint32_t carry = 0;
  for (int64_t base = 0; base < np; base += 4 * kBlock) {
    uint32_t v[4], sum = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = base + 4 * threadIdx.x + u;
      v[u] = k < np ? part[k] : 0u;
      sum += v[u];
    }
    uint32_t tot;
    uint32_t ex = block_excl<uint32_t>(sum, &tot) + carry;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = base + 4 * threadIdx.x + u;
      if (k < np) part[k] = ex;
      ex += v[u];
    }
    carry += tot;
  }
}

// (SELF: `part` holds the chunk sums themselves, not yet scanned; every block
// adds up those before its own, at most kSelfParts of them, in place of
// k_scan_top.)
constexpr int64_t kSelfParts = 4 * kBlock;
template <bool SELF>
__global__ __launch_bounds__(kBlock) void k_scan_apply(uint32_t* __restrict__ a, int64_t n,
                                                       const uint32_t* __restrict__ part) {
  const int64_t base = blockIdx.x * static_cast<int64_t>(kScanChunk) + 4 * threadIdx.x;
  uint32_t v[4], sum = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    v[u] = base + u < n ? a[base + u] : 0u;
    sum += v[u];
  }
  uint32_t pbase;
  if constexpr (SELF) {
    uint32_t pv = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = 4 * threadIdx.x + u;
      pv += k < static_cast<int64_t>(blockIdx.x) ? part[k] : 0u;
    }
    uint32_t ptot;
    block_excl<uint32_t>(pv, &ptot);
    pbase = ptot;
  } else {
    pbase = part[blockIdx.x];
  }
  uint32_t tot;
  uint32_t ex = block_excl<uint32_t>(sum, &tot) + pbase;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (base + u < n) a[base + u] = ex;
    ex += v[u];
  }
}

// ---------------------------------------------------------------------------
// Radix sort passes
// ---------------------------------------------------------------------------
template <int DB>
__global__ __launch_bounds__(kBlock) void k_rs_hist(const uint64_t* __restrict__ keys,
                                                    const DeviceHeader* __restrict__ hdr,
                                                    int shift, int64_t nblocks,
                                                    uint32_t* __restrict__ hist) {
  constexpr int kDig = 1 << DB;
  __shared__ uint32_t s_h[kDig];
  for (int d = threadIdx.x; d < kDig; d += kBlock) s_h[d] = 0;
  __syncthreads();
  const int64_t n = hdr->n_out;
  const int64_t base = blockIdx.x * static_cast<int64_t>(kSortTile);
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int64_t e = base + r * kBlock + threadIdx.x;
    if (e < n) atomicAdd(&s_h[(keys[e] >> shift) & (kDig - 1)], 1u);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < kDig; d += kBlock) hist[d * nblocks + blockIdx.x] = s_h[d];
}

// Stable scatter: the block's elements are taken in their input order, in
// rounds of 256 (round-major, thread-minor); inside a wave equal digits are
// ranked with 8 ballots, across waves and rounds with LDS counters.
template <int DB>
__global__ __launch_bounds__(kBlock) void k_rs_scatter(
    const uint64_t* __restrict__ keys, const int32_t* __restrict__ vals,
    uint64_t* __restrict__ keys_out, int32_t* __restrict__ vals_out,
    const DeviceHeader* __restrict__ hdr, int shift, int64_t nblocks,
    const uint32_t* __restrict__ hist) {
  constexpr int kDig = 1 << DB;
  constexpr int kPer = kDig / kBlock;                // digits per thread
  __shared__ uint32_t s_base[kDig];                  // global offset + running count
  __shared__ uint32_t s_wcnt[kBlock / kWave][kDig];
  const int wave = threadIdx.x / kWave;
  const int64_t n = hdr->n_out;
  const int64_t base = blockIdx.x * static_cast<int64_t>(kSortTile);
#pragma unroll
  for (int j = 0; j < kPer; ++j)
    s_base[threadIdx.x + j * kBlock] = hist[(threadIdx.x + j * kBlock) * nblocks + blockIdx.x];
  for (int r = 0; r < kItems; ++r) {
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w)
#pragma unroll
      for (int j = 0; j < kPer; ++j) s_wcnt[w][threadIdx.x + j * kBlock] = 0;
    __syncthreads();
    const int64_t e = base + r * kBlock + threadIdx.x;
    const bool valid = e < n;
    const uint64_t k = valid ? keys[e] : 0;
    const int32_t v = valid ? vals[e] : 0;
    const uint32_t d = static_cast<uint32_t>((k >> shift) & (kDig - 1));
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < DB; ++b) {
      const uint64_t bal = __ballot((d >> b) & 1u);
      same &= ((d >> b) & 1u) ? bal : ~bal;
    }
    const uint32_t rank = __popcll(same & lanes_below());
    if (valid && rank == 0) s_wcnt[wave][d] = __popcll(same);
    __syncthreads();
    uint32_t before = 0;
    for (int w = 0; w < wave; ++w) before += s_wcnt[w][d];
    const uint32_t pos = s_base[d] + before + rank;
    if (valid) {
      keys_out[pos] = k;
      vals_out[pos] = v;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      uint32_t tot = 0;
#pragma unroll
      for (int w = 0; w < kBlock / kWave; ++w) tot += s_wcnt[w][threadIdx.x + j * kBlock];
      s_base[threadIdx.x + j * kBlock] += tot;
    }
    __syncthreads();
  }
}

}  // namespace

size_t radix_sort_scratch_bytes(int64_t n_cap) {
  const int64_t nblocks = (n_cap + kSortTile - 1) / kSortTile;
  const int64_t nh = nblocks * kMaxDigits;
  const int64_t np = (nh + kScanChunk - 1) / kScanChunk;
  return static_cast<size_t>(nh + np + 64) * sizeof(uint32_t);
}

// Digit width for bits [lo_bit, key_bits): 9 where that takes fewer passes.
int radix_digit_bits(int key_bits, int lo_bit) {
  const int nb = key_bits - lo_bit;
  return (nb + 8) / 9 < (nb + 7) / 8 ? 9 : 8;
}

int radix_sort_passes(int key_bits, int lo_bit) {
  const int nb = key_bits - lo_bit;
  if (nb <= 0) return 0;
  const int db = radix_digit_bits(key_bits, lo_bit);
  return (nb + db - 1) / db;
}

// Sort n = hdr->n_out pairs (n <= n_cap) by bits [lo_bit, key_bits) of the
// key (the bits above key_bits are zero).  Ping-pongs between (keys, vals)
// and (keys_tmp, vals_tmp); returns true when the result ends up in the _tmp
// arrays.
bool radix_sort_pairs(uint64_t* keys, int32_t* vals, uint64_t* keys_tmp, int32_t* vals_tmp,
                      const DeviceHeader* hdr, int64_t n_cap, int key_bits, void* scratch,
                      hipStream_t stream, int lo_bit) {
  if (n_cap <= 0 || key_bits <= lo_bit) return false;
  const int db = radix_digit_bits(key_bits, lo_bit);
  const int64_t nblocks = (n_cap + kSortTile - 1) / kSortTile;
  const int64_t nh = nblocks * (int64_t{1} << db);
  const int64_t np = (nh + kScanChunk - 1) / kScanChunk;
  uint32_t* hist = static_cast<uint32_t*>(scratch);
  uint32_t* part = hist + nh;
  const unsigned gb = static_cast<unsigned>(nblocks);
  bool flipped = false;
  for (int shift = lo_bit; shift < key_bits; shift += db) {
    const uint64_t* ki = flipped ? keys_tmp : keys;
    const int32_t* vi = flipped ? vals_tmp : vals;
    uint64_t* ko = flipped ? keys : keys_tmp;
    int32_t* vo = flipped ? vals : vals_tmp;
    if (db == 9)
      k_rs_hist<9><<<gb, kBlock, 0, stream>>>(ki, hdr, shift, nblocks, hist);
    else
      k_rs_hist<8><<<gb, kBlock, 0, stream>>>(ki, hdr, shift, nblocks, hist);
    k_scan_reduce<<<static_cast<unsigned>(np), kBlock, 0, stream>>>(hist, nh, part);
    if (np <= kSelfParts) {
      k_scan_apply<true><<<static_cast<unsigned>(np), kBlock, 0, stream>>>(hist, nh, part);
    } else {
      k_scan_top<<<1, kBlock, 0, stream>>>(part, np);
      k_scan_apply<false><<<static_cast<unsigned>(np), kBlock, 0, stream>>>(hist, nh, part);
    }
    if (db == 9)
      k_rs_scatter<9><<<gb, kBlock, 0, stream>>>(ki, vi, ko, vo, hdr, shift, nblocks, hist);
    else
      k_rs_scatter<8><<<gb, kBlock, 0, stream>>>(ki, vi, ko, vo, hdr, shift, nblocks, hist);
    flipped = !flipped;
  }
  return flipped;
}

}  // namespace spc
