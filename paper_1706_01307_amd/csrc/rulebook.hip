// Rule-book construction on gfx950 (Section 4 of the paper: map the active
// sites to rows, then list the (input row, output row) pairs of every filter
// offset).  Site maps, chosen per build:
//
// One workgroup (VSC layers of at most 2048 sites on at most 2^18 cells):
//   k_build_small   an LDS occupancy bitmap over Z-ordered cells, ranked by a
//                   popcount prefix (the schedule), neighbours by dilated
//                   arithmetic, G and R_i written directly: one launch.
// Dense grid (grids of up to 2^29 cells and at most ~400 cells per site):
//   every cell of the grid holds 1 + row (0 = empty), cells laid out along
//   the Z-order curve of the sites.
//   k_zero_u32 + k_grid_scatter   clear, then store 1 + r into r's cell
//                                 (range errors; duplicates by CAS, or for
//                                 VSC by the occupied-cell count)
//   k_grid_bits / k_bitscan / k_grid_emit
//                                 occupancy bitmap, its prefix counts, and
//                                 the rows in cell order = the Z-order
//                                 schedule the probe, the compaction and the
//                                 forward walk (up to 2^25 cells no
//                                 k_bitscan: every emitting block adds up the
//                                 block counts before its own; grids of at
//                                 most 2^18 cells: k_grid_emit_self alone,
//                                 the bitmap set by the scatter, every block
//                                 counting the words before its own)
//   k_probe_grid                  per schedule position and offset, one load
//                                 of the neighbour's cell -> gather map
//                                 G[i][p] (1 + input row, 0 if none)
// Hashed (any grid up to 65535 per side):
//   VSC: sorted bricks.  k_site_morton (keys and Morton codes in one pass)
//   and a radix sort order the sites by brick (2^b cells per coordinate; the
//   Morton code's bits above the brick's own); runs of one brick are numbered (k_brick_flags / k_bitscan /
//   k_bricks), each brick inserted once into a hash directory; k_pool_fill
//   writes the bricks' cells into a Z-ordered pool and puts every run in cell
//   order, which completes the Z-order schedule; k_brick_nbrs finds the
//   neighbour bricks of every brick, and k_probe_brick looks up every
//   neighbour with one pool load.
//   SC (and SPCONV_RULEBOOK=table): an open-addressing table of sites,
//   k_insert (pack every site into an order-preserving key; CAS-insert it,
//   range errors, duplicates), k_morton + radix sort for the schedule, and
//   k_probe (hash lookups -> G[i][p]).
// Then
//   k_scan       per offset, exclusive scan of the per-wave pair counts
//   k_compact    per-offset stream compaction of G into R_i, in schedule
//                order (wave ballot + mbcnt, per-wave prefix); on small
//                books every block sums the counts itself (no k_scan)
// except the grouped VSC 3x3x3 grid probe, which counts in a first pass and
// writes G and R_i together in a second (k_probe_grid_g4<false / true>).
// SC (output set = sites with an active input in their receptive field):
//   the input sites go into the grid or table as above, then
//   k_sc_mark    every input marks the output sites it feeds in a bitmap
//                over the output grid (lexicographic linear index); on the
//                grid path fused with the scatter (k_sc_scatter_mark)
//   k_bitsum / k_bitscan / k_sc_emit
//                rank the marked sites by a popcount prefix sum, which
//                numbers the output rows in lexicographic order (small
//                bitmaps: k_sc_emit alone); on the grid path the emission
//                also fills the output grid
//   then the schedule of the output sites (the output grid, or Morton codes
//   and the sort), and probe / scan / compact on input site s*y + o.
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "internal.h"

namespace spc {
namespace {

constexpr int kWave = 64;

struct Extents {
  int32_t e[kMaxD];
};

struct OffsetTable {
  int K;
  int D;
  int32_t f[kMaxD];
  int32_t s[kMaxD];
  int32_t r[kMaxD];     // VSC: (f-1)/2; SC: 0
  int centre;           // VSC: index of the zero offset; SC: -1
};

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int prefix_popc(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0));
}

// Inclusive prefix sum over a wave of 64 lanes.
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    T t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

// Exclusive prefix sum over a 256-thread block; *total receives the sum.
template <typename T>
__device__ __forceinline__ T block_excl_scan(T v, T* total) {
  __shared__ T s_w[kBlock / kWave];
  const int wave = threadIdx.x / kWave;
  T inc = wave_incl_scan(v);
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

// Per-dimension offset o_j - r_j of every filter offset i, in LDS.
__device__ void fill_offsets(const OffsetTable& ot, int16_t (*s_off)[kMaxD]) {
  for (int i = threadIdx.x; i < ot.K; i += blockDim.x) {
    int rem = i;
    for (int j = ot.D - 1; j >= 0; --j) {
      int o = rem % ot.f[j];
      rem /= ot.f[j];
      s_off[i][j] = static_cast<int16_t>(o - ot.r[j]);
    }
  }
}

// Per-block pair counts.  During a probe every wave leaves its count for
// offset i in s_cnt[i][wave]; at the end the block writes, per offset, its
// total (scanned later into the block's base) and the exclusive prefixes of
// waves 1..3 packed in bytes 0..2 (each at most 192), wave 3's own count in
// byte 3 (so bytes 2 + 3 give the total as well).
__device__ void publish_counts(const uint8_t (*s_cnt)[kBlock / kWave], int K,
                               int32_t* __restrict__ blk_cnt, uint32_t* __restrict__ wpre,
                               int64_t nblk, int64_t blk) {
  __syncthreads();
  for (int i = threadIdx.x; i < K; i += kBlock) {
    const uint32_t c0 = s_cnt[i][0], c1 = s_cnt[i][1], c2 = s_cnt[i][2], c3 = s_cnt[i][3];
    blk_cnt[i * nblk + blk] = static_cast<int32_t>(c0 + c1 + c2 + c3);
    wpre[i * nblk + blk] = c0 | ((c0 + c1) << 8) | ((c0 + c1 + c2) << 16) | (c3 << 24);
  }
}

// XCD-aware block order for the probes, whose neighbouring blocks share
// data: workgroup b runs on XCD b % 8, so the blocks that hold output
// positions (the first ceil(n_out / kBlock); an SC output count is known only
// on the device, the launch is sized for a bound) are dealt to the XCDs in
// contiguous ranges, x getting [x * per, (x + 1) * per), and its L2 holds
// that stretch of the schedule's neighbourhood.  The remaining blocks of the
// bound, which only write zeros, follow in order.  The grid must have
// probe_grid_size(nblk) workgroups; returns -1 for a workgroup without a block.
__device__ __forceinline__ int64_t probe_block(int64_t n_rows, int64_t nblk) {
  int64_t nreal = (n_rows + kBlock - 1) / kBlock;
  if (nreal > nblk) nreal = nblk;
  const int64_t per = (nreal + 7) / 8;
  const int64_t L = blockIdx.x;
  if (L < 8 * per) {
    const int64_t b = (L % 8) * per + L / 8;
    return b < nreal ? b : -1;
  }
  const int64_t b = nreal + (L - 8 * per);
  return b < nblk ? b : -1;
}
// 8 ceil(nblk / 8) + 8 >= nblk + 8: the tail covers the blocks past the real
// ones even when the first 8 per slots round up by 7.
inline unsigned probe_grid_size(int64_t nblk) {
  return static_cast<unsigned>(8 * ((nblk + 7) / 8) + 8);
}

__device__ __forceinline__ uint32_t wave_prefix(uint32_t packed, int wave) {
  return wave ? (packed >> (8 * (wave - 1))) & 0xffu : 0u;
}

__global__ void k_fill_u64(uint64_t* __restrict__ p, uint64_t v, uint64_t n) {
  uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
  for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n;
       i += stride)
    p[i] = v;
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint32_t v, uint64_t n) {
  uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
  for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n;
       i += stride)
    p[i] = v;
}

// Zero n 32-bit words at a 16-byte aligned p: 16-byte stores, then the tail.
// With hdr set, also initialises the build's header (status 0, n_out).
__global__ void k_zero_u32(uint32_t* __restrict__ p, uint64_t n, DeviceHeader* hdr,
                           int64_t n_out) {
  const uint64_t n4 = n / 4;
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
  const uint64_t t = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x;
  if (hdr && t == 0) {
    hdr->status = 0;
    hdr->pad = 0;
    hdr->n_out = n_out;
  }
  uint4* q = reinterpret_cast<uint4*>(p);
  for (uint64_t i = t; i < n4; i += stride) q[i] = make_uint4(0u, 0u, 0u, 0u);
  if (t < n - 4 * n4) p[4 * n4 + t] = 0u;
}

__global__ void k_init_header(DeviceHeader* h, int64_t n_out) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    h->status = 0;
    h->pad = 0;
    h->n_out = n_out;
  }
}

// ---------------------------------------------------------------------------
// Small VSC layers (at most kSmallN sites on at most 2^kSmallCellBits cells):
// the whole build in one workgroup, one launch instead of the eight of the
// grid path, whose launch latencies dominate a layer of a few hundred sites.
// Cells are numbered along the Z-order curve (sample on top, then the
// coordinates' bits level by level from the most significant, coordinate 1
// first inside a level); an occupancy bitmap over those cells sits in LDS,
// and the exclusive popcount prefix of its words ranks every occupied cell,
// which is the site's schedule position.  A neighbour lookup is one bit test
// plus that rank.  One wave per (offset, 64 positions) counts the chunk's
// pairs, a block scan of the counts in (offset, chunk) order places every
// chunk's first pair (and so R_i's offset and the bases of its 256-position
// blocks), and a second pass over the chunks writes G and the pairs.
// ---------------------------------------------------------------------------
constexpr int kSmallN = 2048;
constexpr int kSmallThreads = 1024;
constexpr int kSmallCellBits = 18;
constexpr int kSmallWords = (1 << kSmallCellBits) / 32;
constexpr int kSmallK = 128;      // filter offsets (at most 125 = 5^3)

// Coordinate v (< 2^(kSmallCellBits / d)) spread to every d-th bit, d = 1, 2, 3.
__device__ __forceinline__ uint32_t spread_bits(uint32_t v, int d) {
  uint32_t x = v;
  if (d == 2) {
    x = (x | (x << 8)) & 0x00ff00ffu;
    x = (x | (x << 4)) & 0x0f0f0f0fu;
    x = (x | (x << 2)) & 0x33333333u;
    x = (x | (x << 1)) & 0x55555555u;
  } else if (d == 3) {
    x = (x | (x << 16)) & 0xff0000ffu;
    x = (x | (x << 8)) & 0x0300f00fu;
    x = (x | (x << 4)) & 0x030c30c3u;
    x = (x | (x << 2)) & 0x09249249u;
  }
  return x;
}

// Z-order cell of site c (c[0] = sample, c[1..D-1] in range): the spatial
// bits interleaved with coordinate 1 on top inside a level, the sample above
// the sbits spatial bits.
template <int D>
__device__ __forceinline__ uint32_t zcell(const int32_t* c, int sbits) {
  constexpr int d = D - 1;
  uint32_t z = 0;
#pragma unroll
  for (int j = 1; j < D; ++j) z |= spread_bits(static_cast<uint32_t>(c[j]), d) << (D - 1 - j);
  return (static_cast<uint32_t>(c[0]) << sbits) | z;
}

// Moves cell z by a signed offset along the dimension whose bits are m, by
// dilated-integer arithmetic: the field gains (or loses) dz, the spread
// offset, modulo its 2^B values, and the other fields keep their bits.
__device__ __forceinline__ uint32_t zmove(uint32_t z, uint32_t m, uint32_t dz, bool neg) {
  const uint32_t f = neg ? (z & m) - dz : (z | ~m) + dz;
  return (z & ~m) | (f & m);
}

// The cells are numbered with B bits per spatial coordinate, 2^B at least
// extent + (f - 1) / 2 in every dimension, so a neighbour off the grid wraps
// (modulo 2^B) onto a cell past the extent, which no site occupies: no range
// test is needed on the way to the occupancy bit.
template <int D>
__global__ __launch_bounds__(kSmallThreads) void k_build_small(
    const int32_t* __restrict__ coords, int N, int sbits, int nwords, OffsetTable ot, Extents E,
    int32_t* __restrict__ out_coords, int32_t* __restrict__ perm, int32_t* __restrict__ gmap,
    int64_t gstride, int32_t* __restrict__ blk_base, int64_t nblk, int64_t* __restrict__ totals,
    int64_t* __restrict__ pair_off, int2* __restrict__ pairs, DeviceHeader* __restrict__ hdr) {
  constexpr int d = D - 1;
  constexpr int PER = kSmallN / kSmallThreads;     // sites per thread
  constexpr int WPT = kSmallWords / kSmallThreads;  // bitmap words per thread in the scan
  constexpr int NW = kSmallThreads / kWave;
  constexpr int CPT = kSmallK * (kSmallN / kWave) / kSmallThreads;   // chunk counts per thread
  __shared__ uint32_t s_bits[kSmallWords];
  __shared__ uint16_t s_pre[kSmallWords];
  __shared__ int32_t s_row[kSmallN];               // schedule position -> row
  __shared__ uint32_t s_z[kSmallN];                // schedule position -> cell
  __shared__ uint32_t s_dz[kSmallK][kMaxD];        // spread |o_j| of offset i
  __shared__ uint32_t s_neg[kSmallK];              // bit j: o_j < 0
  __shared__ int32_t s_cnt[kSmallK * (kSmallN / kWave)];   // pairs per (offset, 64 positions)
  __shared__ int32_t s_wsum[NW];
  __shared__ uint32_t s_status;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = lane_id();
  const int B = sbits / d;
  uint32_t m[kMaxD] = {0, 0, 0, 0};                // bits of spatial coordinate j
#pragma unroll
  for (int j = 1; j < D; ++j) m[j] = spread_bits((1u << B) - 1u, d) << (D - 1 - j);
  for (int w = tid; w < nwords; w += kSmallThreads) s_bits[w] = 0;
  for (int p = tid; p < kSmallN; p += kSmallThreads) {
    s_row[p] = 0;
    s_z[p] = 0;
  }
  for (int i = tid; i < ot.K; i += kSmallThreads) {
    int rem = i;
    uint32_t neg = 0;
#pragma unroll
    for (int j = D - 1; j >= 0; --j) {
      const int o = rem % ot.f[j] - ot.r[j];
      rem /= ot.f[j];
      s_dz[i][j] = j > 0 ? spread_bits(static_cast<uint32_t>(o < 0 ? -o : o), d) << (D - 1 - j) : 0u;
      neg |= static_cast<uint32_t>(o < 0) << j;
    }
    s_neg[i] = neg;
  }
  if (tid == 0) s_status = 0;
  __syncthreads();
  // Block-wide exclusive scan of one value per thread; *total = the sum.
  auto block_scan = [&](int v, int* total) {
    const int inc = wave_incl_scan(v);
    if (lane == kWave - 1) s_wsum[wave] = inc;
    __syncthreads();
    int ex = inc - v, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (w < wave) ex += s_wsum[w];
      tot += s_wsum[w];
    }
    __syncthreads();
    *total = tot;
    return ex;
  };
  // 1. every site sets its cell's bit (a bit already set: a duplicate site;
  // a coordinate out of range: status, and no cell)
  uint32_t cell[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int p = tid + u * kSmallThreads;
    cell[u] = ~0u;
    if (p < N) {
      int32_t c[kMaxD] = {0, 0, 0, 0};
      bool ok = true;
#pragma unroll
      for (int j = 0; j < D; ++j) {
        c[j] = coords[static_cast<int64_t>(p) * D + j];
        out_coords[static_cast<int64_t>(p) * D + j] = c[j];
        ok = ok && c[j] >= 0 && c[j] < E.e[j];
      }
      if (ok) {
        cell[u] = zcell<D>(c, sbits);
        const uint32_t bit = 1u << (cell[u] & 31);
        if (atomicOr(&s_bits[cell[u] >> 5], bit) & bit) atomicOr(&s_status, kStDup);
      } else {
        atomicOr(&s_status, kStRange);
      }
    }
  }
  __syncthreads();
  // 2. exclusive prefix of the words' popcounts (each thread WPT words)
  {
    uint32_t cnt[WPT];
    int sum = 0;
#pragma unroll
    for (int k = 0; k < WPT; ++k) {
      const int w = tid * WPT + k;
      cnt[k] = w < nwords ? __popc(s_bits[w]) : 0u;
      sum += static_cast<int>(cnt[k]);
    }
    int tot;
    int ex = block_scan(sum, &tot);
#pragma unroll
    for (int k = 0; k < WPT; ++k) {
      const int w = tid * WPT + k;
      if (w < nwords) s_pre[w] = static_cast<uint16_t>(ex);
      ex += static_cast<int>(cnt[k]);
    }
  }
  __syncthreads();
  // 3. the rank of a site's cell is its schedule position
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (cell[u] == ~0u) continue;
    const uint32_t w = cell[u] >> 5;
    const int pos = s_pre[w] + __popc(s_bits[w] & ((1u << (cell[u] & 31)) - 1u));
    s_row[pos] = tid + u * kSmallThreads;
    s_z[pos] = cell[u];
  }
  __syncthreads();
  for (int p = tid; p < N; p += kSmallThreads) perm[p] = s_row[p];
  // Neighbour of schedule position p at offset i: 1 + its row, 0 if none.
  // With RANK false only whether there is one (0 / 1).
  auto neighbour = [&](int p, int i, auto rank) -> int32_t {
    uint32_t z = s_z[p];
    const uint32_t neg = s_neg[i];
#pragma unroll
    for (int j = 1; j < D; ++j) z = zmove(z, m[j], s_dz[i][j], (neg >> j) & 1u);
    const uint32_t word = s_bits[z >> 5];
    const uint32_t bit = 1u << (z & 31);
    if (!(word & bit)) return 0;
    if constexpr (!decltype(rank)::value) return 1;
    else return s_row[s_pre[z >> 5] + __popc(word & (bit - 1u))] + 1;
  };
  // Visits the (offset, chunk of 64 positions) tasks of nchunk chunks per
  // offset, wave by wave in steps of NW, without a division per task.
  auto for_tasks = [&](int nchunk, auto fn) {
    if (nchunk == 0) return;
    int i = wave / nchunk, c = wave % nchunk;
    for (; i < ot.K;) {
      fn(i, c);
      c += NW;
      while (c >= nchunk) {
        c -= nchunk;
        ++i;
      }
    }
  };
  // 4. pairs per (offset, chunk of 64 positions), one wave per chunk
  const int nch = (N + kWave - 1) / kWave;
  const int ntask = ot.K * nch;
  for_tasks(nch, [&](int i, int c) {
    const int p = c * kWave + lane;
    const bool hit = p < N && neighbour(p, i, std::false_type{});
    const int n = __popcll(__ballot(hit));
    if (lane == 0) s_cnt[i * nch + c] = n;
  });
  __syncthreads();
  // 5. exclusive scan of the chunk counts in (offset, chunk) order: the first
  // pair of every chunk
  int tot;
  {
    int v[CPT], sum = 0;
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int t = tid * CPT + k;
      v[k] = t < ntask ? s_cnt[t] : 0;
      sum += v[k];
    }
    int ex = block_scan(sum, &tot);
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int t = tid * CPT + k;
      if (t < ntask) s_cnt[t] = ex;
      ex += v[k];
    }
  }
  __syncthreads();
  for (int i = tid; i < ot.K; i += kSmallThreads) {
    const int first = s_cnt[i * nch];
    pair_off[i] = first;
    totals[i] = (i + 1 < ot.K ? s_cnt[(i + 1) * nch] : tot) - first;
  }
  for (int t = tid; t < ot.K * nblk; t += kSmallThreads) {
    const int i = static_cast<int>(t / nblk), b = static_cast<int>(t % nblk);
    blk_base[t] = s_cnt[i * nch + b * (kBlock / kWave)] - s_cnt[i * nch];
  }
  // 6. gather map (zeros up to the padded stride) and pairs, one wave per chunk
  for_tasks(static_cast<int>(gstride / kWave), [&](int i, int c) {
    const int p = c * kWave + lane;
    const int32_t e = p < N ? neighbour(p, i, std::true_type{}) : 0;
    gmap[static_cast<int64_t>(i) * gstride + p] = e;
    const uint64_t mk = __ballot(e != 0);
    if (e) pairs[s_cnt[i * nch + c] + prefix_popc(mk)] = make_int2(e - 1, s_row[p]);
  });
  if (tid == 0) {
    pair_off[ot.K] = tot;
    hdr->status = s_status;
    hdr->pad = 0;
    hdr->n_out = N;
  }
}

// Insert input row r's site into the table.
template <bool WIDE>
__global__ __launch_bounds__(kBlock) void k_insert(
    const int32_t* __restrict__ coords, int64_t N, Codec c, Table t,
    uint64_t* __restrict__ keys, int32_t* __restrict__ copy_out,
    uint32_t* __restrict__ status) {
  const int64_t r = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (r >= N) return;
  int32_t x[kMaxD];
  bool ok = true;
  for (int j = 0; j < c.D; ++j) {
    x[j] = coords[r * c.D + j];
    ok = ok && x[j] >= 0 && x[j] < c.size[j];
    if (copy_out) copy_out[r * c.D + j] = x[j];
  }
  if (!ok) {
    keys[r] = kEmpty;
    atomicOr(status, kStRange);
    return;
  }
  const uint64_t key = pack_site(c, x);
  keys[r] = key;
  const uint64_t entry = WIDE ? key : (key << t.rbits) | static_cast<uint64_t>(r);
  uint64_t b = home_bucket(t, key);
  for (uint64_t p = 0; p < t.nbuckets; ++p) {
    uint64_t* B = t.slots + 4 * b;
    for (int j = 0; j < 4; ++j) {
      // CAS straight away (at a quarter load the first try usually wins); a
      // failed CAS returns the occupant, which decides duplicate or move on
      const uint64_t cur = atomicCAS(reinterpret_cast<unsigned long long*>(&B[j]),
                                     static_cast<unsigned long long>(kEmpty),
                                     static_cast<unsigned long long>(entry));
      if (cur == kEmpty) {
        if (WIDE) t.vals[4 * b + j] = static_cast<int32_t>(r);
        return;
      }
      const bool same = WIDE ? (cur == key) : ((cur >> t.rbits) == key);
      if (same) {
        atomicOr(status, kStDup);
        return;
      }
    }
    b = (b + 1) & (t.nbuckets - 1);
  }
  atomicOr(status, kStCap);
}

// Neighbour probe.  Row y's site is unpacked from rowkeys[y] with `crow`; the
// site feeding it through offset i is y + o_i - r (VSC) or s*y + o_i (SC),
// packed with `cin` and looked up in the input table.  Offsets go in batches
// of 8 and every bucket load of a batch is issued unconditionally (lanes
// whose neighbour is off the grid read some valid bucket and ignore it), so
// 8 loads per thread are in flight at once; a load under a divergent branch
// would instead be waited for on its own.
template <bool WIDE, bool SC, int D>
__global__ __launch_bounds__(kBlock) void k_probe(
    const uint64_t* __restrict__ rowkeys, const int32_t* __restrict__ perm,
    const DeviceHeader* __restrict__ hdr, int64_t gstride, Codec crow, Codec cin, Table t,
    OffsetTable ot, int32_t* __restrict__ gmap, int32_t* __restrict__ blk_cnt,
    uint32_t* __restrict__ wpre, int64_t nblk) {
  const int64_t blk = probe_block(hdr->n_out, nblk);
  if (blk < 0) return;
  __shared__ int16_t s_off[kMaxK][kMaxD];
  __shared__ uint8_t s_cnt[kMaxK][kBlock / kWave];
  fill_offsets(ot, s_off);
  __syncthreads();

  // thread = schedule position p; its output row is perm[p]
  const int64_t n_rows = hdr->n_out;
  const int64_t p = blk * kBlock + threadIdx.x;
  const bool valid = p < n_rows;
  const int wave = threadIdx.x / kWave;
  const int32_t y = valid ? perm[p] : 0;
  const uint64_t rk = rowkeys[y];
  int32_t c[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    c[j] = static_cast<int32_t>((rk >> crow.shift[j]) & crow.fmask[j]);
    if (SC) c[j] *= ot.s[j];
  }

  constexpr int B = 8;
  for (int i0 = 0; i0 < ot.K; i0 += B) {
    uint64_t key[B], bk[B];
    uint64_t sl[B][4];
    bool inb[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int i = i0 + u;
      const int ic = i < ot.K ? i : ot.K - 1;
      bool ok = valid && i < ot.K && i != ot.centre;
      uint64_t k = 0;
#pragma unroll
      for (int j = 0; j < D; ++j) {
        const int32_t n = c[j] + s_off[ic][j];
        ok = ok && n >= 0 && n < cin.size[j];
        k |= static_cast<uint64_t>(static_cast<uint32_t>(n) & cin.fmask[j]) << cin.shift[j];
      }
      key[u] = k;
      inb[u] = ok;
      bk[u] = home_bucket(t, k);
      load_bucket(t, bk[u], sl[u]);
    }
    int32_t r[B];
    bool more = false;
#pragma unroll
    for (int u = 0; u < B; ++u) {
      r[u] = match_bucket<WIDE>(t, bk[u], sl[u], key[u]);
      more = more || (inb[u] && r[u] == -2);
    }
    // Home buckets that were full without the key: one more batched round on
    // the next bucket for the whole wave, then (very rarely) a serial walk.
    if (__ballot(more) != 0) {
#pragma unroll
      for (int u = 0; u < B; ++u) {
        bk[u] = (bk[u] + 1) & (t.nbuckets - 1);
        load_bucket(t, bk[u], sl[u]);
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int32_t r2 = match_bucket<WIDE>(t, bk[u], sl[u], key[u]);
        r[u] = r[u] == -2 ? r2 : r[u];
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int i = i0 + u;
      if (i >= ot.K) break;
      int32_t row = inb[u] ? r[u] : ((valid && i == ot.centre) ? y : -1);
      if (inb[u] && r[u] == -2) row = find_from<WIDE>(t, bk[u], key[u]);
      if (p < gstride) gmap[i * gstride + p] = row + 1;   // 0 = no input
      const uint64_t m = __ballot(row >= 0);
      if (lane_id() == 0) s_cnt[i][wave] = static_cast<uint8_t>(__popcll(m));
    }
  }
  publish_counts(s_cnt, ot.K, blk_cnt, wpre, nblk, blk);
}

// ---------------------------------------------------------------------------
// Sorted-brick site map (VSC layers on grids too large or too sparse for the
// dense grid).  A site's cell is its Z-order code (the Morton code the
// schedule sorts: sample on top, then the coordinates' bits level by level);
// its lowest lb bits, levels 0 .. b-1, place it inside a brick, an aligned
// block of 2^b_j cells along coordinate j.  In the sorted order the sites of
// a brick are one run, so the runs number the occupied bricks in Z-order.  A
// hash directory maps a brick (cell >> lb) to its number, inserted once per
// brick (no two inserts of one key, hence no contention), and a pool holds
// 2^lb entries per brick (1 + row, 0 = empty), bricks in Z-order: a compacted
// Z-ordered grid.  A lookup is a pool load at the brick found in the
// directory; a brick of side 2^b_j >= f_j - 1 lets the neighbours of a site
// touch at most 2^d bricks, whose directory entries the probe fetches once
// per site, all at once.
// ---------------------------------------------------------------------------
constexpr int kBrickK = 128;         // offsets the brick probe takes (5^3 = 125)
constexpr int kBrickCells = 64;      // cells per brick, at most

struct BrickMap {
  ulonglong2* dir;       // directory slots: x = brick (kEmpty = free), y = brick number
  uint64_t dslots;       // allocated slots (power of two)
  int32_t* pool;         // [bricks][2^lb] 1 + row, 0 = empty
  int lb;                // cell bits inside a brick
  int D;
  uint64_t M[kMaxD];     // cell bits of spatial coordinate j
  uint64_t BM[kMaxD];    // brick-number bits of coordinate j (M[j] above lb, shifted down)
  int32_t side[kMaxD];   // 2^b_j
  const DeviceHeader* nbricks;   // n_out = occupied bricks (device)
};

// Directory size in use: a power of two >= 2 x bricks (at least 64) within
// the allocation, so the table is at most half full.
__device__ __forceinline__ uint64_t dir_mask(const BrickMap& m) {
  const uint64_t need = 2 * static_cast<uint64_t>(m.nbricks->n_out);
  const uint64_t want = need > 64 ? 1ull << (64 - __clzll(need - 1)) : 64;
  return (want < m.dslots ? want : m.dslots) - 1;
}

// Slow path of a directory lookup: on from the slot after `sl` (the first
// slot held another brick).
__device__ __noinline__ int32_t dir_find_after(const BrickMap& m, uint64_t dmask, uint64_t sl,
                                               uint64_t key) {
  for (uint64_t t = 0; t < dmask; ++t) {
    sl = (sl + 1) & dmask;
    const ulonglong2 v = m.dir[sl];
    if (v.x == key) return static_cast<int32_t>(v.y);
    if (v.x == kEmpty) return -1;
  }
  return -1;
}

__device__ __forceinline__ uint64_t zmove64(uint64_t z, uint64_t m, uint64_t dz, bool neg) {
  const uint64_t f = neg ? (z & m) - dz : (z | ~m) + dz;
  return (z & ~m) | (f & m);
}

// Bits of v spread over the set bits of m, lowest first.
__host__ __device__ inline uint64_t deposit64(uint64_t v, uint64_t m) {
  uint64_t r = 0;
  for (uint64_t bb = 1; m; bb <<= 1) {
    const uint64_t low = m & (0ull - m);
    if (v & bb) r |= low;
    m &= m - 1;
  }
  return r;
}

// Bits of v at the set positions of m, packed from the lowest.
__device__ __forceinline__ uint32_t extract_bits(uint32_t v, uint32_t m) {
  uint32_t r = 0;
  for (uint32_t bb = 1; m; bb <<= 1) {
    const uint32_t low = m & (0u - m);
    if (v & low) r |= bb;
    m &= m - 1;
  }
  return r;
}

// Entry e = l * K + i of the bricks' neighbourhood table: for a site at
// local cell l (the lowest lb bits of its cell) and offset i, the
// neighbour's local cell | (the faces it crossed, bit j-1 for coordinate j)
// << 6.  The same for every brick, so one small table serves the probe.
__device__ uint16_t brick_table_entry(const OffsetTable& ot, const BrickMap& m, int e) {
  const uint32_t lowmask = (1u << m.lb) - 1u;
  const int l = e / ot.K, i = e % ot.K;
  int rem = i;
  int o[kMaxD] = {0, 0, 0, 0};
  for (int j = m.D - 1; j >= 0; --j) {
    o[j] = rem % ot.f[j] - ot.r[j];
    rem /= ot.f[j];
  }
  uint32_t loc = 0, S = 0;
  for (int j = 1; j < m.D; ++j) {
    const uint32_t lm = static_cast<uint32_t>(m.M[j]) & lowmask;
    int v = static_cast<int>(extract_bits(static_cast<uint32_t>(l), lm)) + o[j];
    if (v < 0 || v >= m.side[j]) {
      S |= 1u << (j - 1);
      v = v < 0 ? v + m.side[j] : v - m.side[j];
    }
    loc |= static_cast<uint32_t>(deposit64(static_cast<uint64_t>(v), lm));
  }
  return static_cast<uint16_t>(loc | (S << 6));
}

// Per sorted position: first of its brick?  The block's flags as four 64-bit
// wave masks and their count; equal cells next to each other are duplicate
// sites; a second mask marks the positions whose rows are in range.  Rows
// out of range (key kEmpty) take part in nothing.  The first
// 2^lb K threads also write the neighbourhood table (the grid has at least
// that many; blocks past the nblk of positions do only that).
__global__ __launch_bounds__(kBlock) void k_brick_flags(
    const uint64_t* __restrict__ mk, const int32_t* __restrict__ perm,
    const uint64_t* __restrict__ rowkeys, int64_t n, int64_t nblk, int lb,
    uint64_t* __restrict__ flagbits, uint64_t* __restrict__ validbits, uint32_t* __restrict__ bsum,
    uint32_t* __restrict__ status, OffsetTable ot, BrickMap bm, uint16_t* __restrict__ tab) {
  __shared__ uint32_t s_c[kBlock / kWave];
  const int64_t p = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (p < (int64_t{1} << bm.lb) * ot.K) tab[p] = brick_table_entry(ot, bm, static_cast<int>(p));
  if (blockIdx.x >= nblk) return;
  const int wave = threadIdx.x / kWave;
  bool flag = false;
  const bool valid = p < n && rowkeys[perm[p]] != kEmpty;
  if (valid) {
    const uint64_t key = mk[p];
    flag = true;
    if (p > 0 && rowkeys[perm[p - 1]] != kEmpty) {
      const uint64_t pk = mk[p - 1];
      flag = (pk >> lb) != (key >> lb);
      if (pk == key) atomicOr(status, kStDup);
    }
  }
  const uint64_t m = __ballot(flag);
  const uint64_t mv = __ballot(valid);
  if (lane_id() == 0) {
    flagbits[p >> 6] = m;
    validbits[p >> 6] = mv;
    s_c[wave] = static_cast<uint32_t>(__popcll(m));
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kBlock / kWave; ++w) t += s_c[w];
    bsum[blockIdx.x] = t;
  }
}

// Brick number of every sorted position (its brick's rank among the flags);
// the first position of a brick inserts it into the directory and records
// where its run starts.
__global__ __launch_bounds__(kBlock) void k_bricks(
    const uint64_t* __restrict__ mk, const int32_t* __restrict__ perm,
    int64_t n, const uint64_t* __restrict__ flagbits, const uint64_t* __restrict__ validbits,
    const uint32_t* __restrict__ bbase, BrickMap m, int32_t* __restrict__ brickidx,
    int64_t* __restrict__ starts) {
  const int64_t p = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (p >= n) return;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const uint64_t w64 = flagbits[p >> 6];
  uint32_t before = bbase[blockIdx.x];
  for (int w = 0; w < wave; ++w) before += __popcll(flagbits[(blockIdx.x * (kBlock / kWave)) + w]);
  const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);
  const int64_t bi = static_cast<int64_t>(before) + __popcll(w64 & upto) - 1;
  const bool valid = (validbits[p >> 6] >> lane) & 1ull;
  brickidx[p] = valid ? static_cast<int32_t>(bi) : -1;
  if (!((w64 >> lane) & 1ull)) return;
  starts[bi] = p;
  const uint64_t brick = mk[p] >> m.lb;
  const uint64_t dmask = dir_mask(m);
  uint64_t sl = mix64(brick) & dmask;
  for (uint64_t t = 0; t <= dmask; ++t) {
    const uint64_t old = atomicCAS(reinterpret_cast<unsigned long long*>(&m.dir[sl].x),
                                   static_cast<unsigned long long>(kEmpty),
                                   static_cast<unsigned long long>(brick));
    if (old == kEmpty) {
      m.dir[sl].y = static_cast<uint64_t>(bi);
      break;
    }
    if (old == brick) break;          // (only after an out-of-range site split a run)
    sl = (sl + 1) & dmask;
  }
}

// Pool entries of every brick, one wave per brick (bricks dealt out in steps
// of the grid's waves): the run's sites go into an LDS image of the brick,
// which the wave then stores whole (zeros included) in one coalesced pass.
// The schedule was sorted by brick only: the occupied cells of the image, in
// cell order, are the run's sites in Morton order, and the wave writes them
// back over the run (codes and rows).  Two sites on one cell are duplicates.
constexpr int kPoolBlocks = 2048;
__global__ __launch_bounds__(kBlock) void k_pool_fill(
    uint64_t* __restrict__ mk, int32_t* __restrict__ perm,
    const uint64_t* __restrict__ validbits, int64_t n, const int64_t* __restrict__ starts,
    BrickMap m, uint32_t* __restrict__ status) {
  __shared__ int32_t s_img[kBlock / kWave][kBrickCells];
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int64_t nbr = m.nbricks->n_out;
  const int cells = 1 << m.lb;
  const uint64_t lowmask = static_cast<uint64_t>(cells - 1);
  const int64_t nw = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
  bool dup = false;
  // the next brick's run bounds are requested while this brick is filled
  int64_t bi = blockIdx.x * static_cast<int64_t>(kBlock / kWave) + wave;
  int64_t nfirst = bi < nbr ? starts[bi] : 0;
  int64_t nlast = bi + 1 < nbr ? starts[bi + 1] : n;
  for (; bi < nbr; bi += nw) {
    const int64_t first = nfirst, last = nlast;
    const int64_t bn = bi + nw;
    nfirst = bn < nbr ? starts[bn] : 0;
    nlast = bn + 1 < nbr ? starts[bn + 1] : n;
    const uint64_t brick = mk[first] >> m.lb;      // a run starts on a site in range
    s_img[wave][lane] = 0;
    for (int64_t q0 = first; q0 < last; q0 += kWave) {
      const int64_t q = q0 + lane;
      if (q < last && ((validbits[q >> 6] >> (q & 63)) & 1ull))
        dup |= atomicExch(&s_img[wave][mk[q] & lowmask], perm[q] + 1) != 0;
    }
    const int32_t v = lane < cells ? s_img[wave][lane] : 0;
    if (lane < cells) m.pool[(bi << m.lb) + lane] = v;
    const uint64_t occ = __ballot(v != 0);
    if (v != 0) {
      const int64_t pos = first + __popcll(occ & ((1ull << lane) - 1));
      perm[pos] = v - 1;
      mk[pos] = (brick << m.lb) | static_cast<uint64_t>(lane);
    }
  }
  if (dup) atomicOr(status, kStDup);
}

// Neighbour bricks of every brick: entry [bi][t] = the number of the brick
// at brick offset t (digit j-1 of t in base 3 = the step along coordinate j
// plus one), -1 if absent or off the grid, so the probe, whose sites read
// their brick's row, hashes nothing.  One thread per (brick, offset in the
// upper half t >= NB/2): brick B at offset t of brick A has A at offset
// NB-1-t, so each lookup fills both entries (the lower halves start at -1,
// cleared with the directory).  Pairs are dealt out in steps of the grid.
__global__ __launch_bounds__(kBlock) void k_brick_nbrs(
    const uint64_t* __restrict__ mk, const int64_t* __restrict__ starts, Codec crow, BrickMap m,
    int nb3, int32_t* __restrict__ nbr) {
  const int half = nb3 / 2;
  const int per = nb3 - half;                 // offsets half .. nb3-1
  const int64_t total = m.nbricks->n_out * per;
  const uint64_t dmask = dir_mask(m);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; e < total;
       e += stride) {
    const int64_t bi = e / per;
    const int t0 = half + static_cast<int>(e - bi * per);
    if (t0 == half) {                         // the brick itself
      nbr[bi * nb3 + half] = static_cast<int32_t>(bi);
      continue;
    }
    const int64_t p = starts[bi];
    // the brick's coordinates are the brick-number bits of its key (no trip
    // through the row's packed key)
    const uint64_t k0 = mk[p] >> m.lb;
    uint64_t k = k0;
    bool ok = true;
    int t = t0;
    for (int j = 1; j < m.D; ++j) {
      const int dj = t % 3 - 1;
      t /= 3;
      if (dj == 0) continue;
      uint64_t bj = 0, bm = m.BM[j];              // bits of k0 at BM[j], packed from the lowest
      for (uint64_t bb = 1; bm; bb <<= 1) {
        if (k0 & bm & (0ull - bm)) bj |= bb;
        bm &= bm - 1;
      }
      const int32_t bc = static_cast<int32_t>(bj) + dj, bmax = (crow.size[j] - 1) / m.side[j];
      ok = ok && m.BM[j] != 0 && bc >= 0 && bc <= bmax;
      k = zmove64(k, m.BM[j], m.BM[j] & (0ull - m.BM[j]), dj < 0);
    }
    int32_t r = -1;
    if (ok) {
      const uint64_t sl = mix64(k) & dmask;
      const ulonglong2 v = m.dir[sl];
      if (v.x == k) r = static_cast<int32_t>(v.y);
      else if (v.x != kEmpty) r = dir_find_after(m, dmask, sl, k);
    }
    nbr[bi * nb3 + t0] = r;
    if (r >= 0) nbr[static_cast<int64_t>(r) * nb3 + (nb3 - 1 - t0)] = static_cast<int32_t>(bi);
  }
}

// Clears the directory slots in use (dir_mask), kEmpty in both halves, and
// sets the bricks' neighbour rows to -1.
__global__ __launch_bounds__(kBlock) void k_dir_clear(BrickMap m, int32_t* __restrict__ nbr,
                                                      int nb3) {
  const uint64_t n = dir_mask(m) + 1;
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
  for (uint64_t i = blockIdx.x * static_cast<uint64_t>(kBlock) + threadIdx.x; i < n; i += stride)
    m.dir[i] = make_ulonglong2(kEmpty, kEmpty);
  const uint64_t nn = static_cast<uint64_t>(m.nbricks->n_out) * nb3;
  for (uint64_t i = blockIdx.x * static_cast<uint64_t>(kBlock) + threadIdx.x; i < nn; i += stride)
    nbr[i] = -1;
}

// Neighbour probe on the brick map (VSC).  Thread = sorted position p, which
// is the schedule position; its cell is mk[p].  The bricks the neighbours can
// fall in are the site's own and, per coordinate where the site lies within
// (f-1)/2 of its brick's face, the brick across that face (none where that
// face is the grid's): at most 2^(D-1) combinations, whose directory slots
// are loaded together before any pool load.  The neighbourhood table gives
// each offset's local cell and combination, so a lookup is one LDS read, a
// select and one pool load; a neighbour past an extent lands on a cell no
// site occupies.
template <int D>
__global__ __launch_bounds__(kBlock) void k_probe_brick(
    const uint64_t* __restrict__ mk, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ brickidx, const uint64_t* __restrict__ rowkeys,
    const DeviceHeader* __restrict__ hdr, int64_t gstride, Codec crow, OffsetTable ot,
    BrickMap m, const uint16_t* __restrict__ tab, const int32_t* __restrict__ nbr, int nb3,
    int32_t* __restrict__ gmap, int32_t* __restrict__ blk_cnt, uint32_t* __restrict__ wpre,
    int64_t nblk) {
  const int64_t blk = probe_block(hdr->n_out, nblk);
  if (blk < 0) return;
  constexpr int NS = 1 << (D - 1);    // brick combinations
  __shared__ uint16_t s_tab[kBrickCells * kBrickK];
  __shared__ uint8_t s_cnt[kBrickK][kBlock / kWave];
  const int ntab = (1 << m.lb) * ot.K;
  for (int e = threadIdx.x; e < ntab; e += kBlock) s_tab[e] = tab[e];
  __syncthreads();

  const int64_t n_rows = hdr->n_out;
  const int64_t p = blk * kBlock + threadIdx.x;
  const bool valid = p < n_rows && brickidx[p] >= 0;
  const int wave = threadIdx.x / kWave;
  const int32_t y = p < n_rows ? perm[p] : 0;
  const uint64_t cell0 = p < n_rows ? mk[p] : 0;
  const uint64_t rk = rowkeys[y];
  const uint64_t lowmask = (1ull << m.lb) - 1;
  // per coordinate: the face the neighbours can cross (e = -1 / +1, 0 none),
  // 0 as well where the brick across it would be off the grid
  int e[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    e[j] = 0;
    if (j > 0 && m.BM[j] != 0) {
      const int32_t c = static_cast<int32_t>((rk >> crow.shift[j]) & crow.fmask[j]);
      const int low = c & (m.side[j] - 1);
      const int32_t bc = c / m.side[j], bmax = (crow.size[j] - 1) / m.side[j];
      if (low < ot.r[j] && bc > 0) e[j] = -1;
      else if (low >= m.side[j] - ot.r[j] && bc < bmax) e[j] = 1;
    }
  }
  // the site's brick row of the neighbour table: combination S of the faces
  // the site can cross is brick offset sum_j (S_j ? e_j + 1 : 1) 3^(j-1)
  const int64_t brow = static_cast<int64_t>(valid ? brickidx[p] : 0) * nb3;
  int32_t idx[NS];
  idx[0] = valid ? brickidx[p] : -1;
#pragma unroll
  for (int S = 1; S < NS; ++S) {
    bool need = valid;
    int t = 0, w = 1;
#pragma unroll
    for (int j = 1; j < D; ++j) {
      const bool in = (S >> (j - 1)) & 1;
      need = need && (!in || e[j] != 0);
      t += (in ? e[j] + 1 : 1) * w;
      w *= 3;
    }
    const int32_t r = nbr[brow + (need ? t : 0)];    // every load in flight at once
    idx[S] = need ? r : -1;
  }
  const int lrow = static_cast<int>(cell0 & lowmask) * ot.K;

  constexpr int B = 8;
  for (int i0 = 0; i0 < ot.K; i0 += B) {
    int32_t v[B];
    bool ok[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int i = i0 + u;
      const uint32_t t = s_tab[lrow + (i < ot.K ? i : 0)];
      const uint32_t S = t >> 6;
      int32_t b = idx[0];
#pragma unroll
      for (int q = 1; q < NS; ++q) b = S == static_cast<uint32_t>(q) ? idx[q] : b;
      ok[u] = valid && i < ot.K && b >= 0;
      const int64_t a = ok[u] ? (static_cast<int64_t>(b) << m.lb) + (t & 63u) : 0;
      v[u] = m.pool[a];                   // unconditional: entry 0 exists
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int i = i0 + u;
      if (i >= ot.K) break;
      const int32_t row = ok[u] ? v[u] - 1 : -1;
      if (p < gstride) gmap[i * gstride + p] = row + 1;   // 0 = no input
      const uint64_t mm = __ballot(row >= 0);
      if (lane_id() == 0) s_cnt[i][wave] = static_cast<uint8_t>(__popcll(mm));
    }
  }
  publish_counts(s_cnt, ot.K, blk_cnt, wpre, nblk, blk);
}

// One block per offset: exclusive scan of its per-block counts, in place;
// total into totals[i].
__global__ __launch_bounds__(kBlock) void k_scan(int32_t* __restrict__ blk_cnt, int64_t nblk,
                                                 int64_t* __restrict__ totals) {
  // 16 counts per thread, all requested at once: one round of load latency
  // per 4,096 blocks (the headline's 3,526 blocks in one)
  constexpr int PER = 16;
  int32_t* c = blk_cnt + blockIdx.x * nblk;
  int64_t carry = 0;
  for (int64_t base = 0; base < nblk; base += PER * kBlock) {
    int32_t v[PER];
    int64_t sum = 0;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t k = base + PER * threadIdx.x + u;
      v[u] = k < nblk ? c[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) sum += v[u];
    int64_t tot;
    int64_t ex = block_excl_scan<int64_t>(sum, &tot) + carry;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t k = base + PER * threadIdx.x + u;
      if (k < nblk) c[k] = static_cast<int32_t>(ex);
      ex += v[u];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// Compaction of the gather map into the per-offset pair lists: every wave
// writes its pairs of offset i at pair_off[i] + (pairs of the blocks before
// it) + (pairs of the waves before it in its block) + (set lanes before it in
// its ballot), so R_i comes out in schedule (Z-order) order without any
// further sorting.  SELF: no k_scan ran; every block sums the probe's counts
// (from the packed wave prefixes) of all blocks itself, for k_i and for its
// own base, which it stores in blk_base (small books: K nblk^2 words read).
template <bool SELF>
__global__ __launch_bounds__(kBlock) void k_compact(
    const int32_t* __restrict__ gmap, const int32_t* __restrict__ perm,
    int32_t* __restrict__ blk_base, const uint32_t* __restrict__ wpre,
    int64_t* __restrict__ totals, int K, int64_t gstride, int64_t n_cap,
    const DeviceHeader* __restrict__ hdr, int64_t nblk, int2* __restrict__ pairs,
    int64_t* __restrict__ pair_off) {
  __shared__ int64_t s_off[kMaxK + 1];
  __shared__ uint32_t s_wp[kMaxK];
  __shared__ int64_t s_tot[SELF ? kMaxK : 1];
  __shared__ int32_t s_base[SELF ? kMaxK : 1];
  // the gather-map entries of the first kCompactPre offsets and the output
  // row, requested before anything else so that their latency passes during
  // the block's prefix work (p < gstride: in bounds; positions past the
  // output rows are dropped below)
  constexpr int kCompactPre = 16;
  const int64_t p = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  int32_t pre[kCompactPre];
#pragma unroll
  for (int u = 0; u < kCompactPre; ++u)
    pre[u] = gmap[(u < K ? u : K - 1) * gstride + p] - 1;
  const int32_t y0 = perm[p < n_cap ? p : 0];
  if constexpr (SELF) {
    const int wave = threadIdx.x / kWave, lane = lane_id();
    for (int k = wave; k < K; k += kBlock / kWave) {
      int64_t tot = 0, base = 0;
      for (int64_t b = lane; b < nblk; b += kWave) {
        const uint32_t w = wpre[k * nblk + b];
        const int64_t c = ((w >> 16) & 0xffu) + (w >> 24);
        tot += c;
        base += b < static_cast<int64_t>(blockIdx.x) ? c : 0;
      }
      tot = __shfl(wave_incl_scan(tot), kWave - 1, kWave);
      base = __shfl(wave_incl_scan(base), kWave - 1, kWave);
      if (lane == 0) {
        s_tot[k] = tot;
        s_base[k] = static_cast<int32_t>(base);
      }
    }
    __syncthreads();
  }
  // pair_off = exclusive prefix of totals (K <= 1024, 4 per thread).
  {
    int64_t v[4], sum = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = 4 * threadIdx.x + u;
      v[u] = k < K ? (SELF ? s_tot[k] : totals[k]) : 0;
      sum += v[u];
    }
    int64_t tot;
    int64_t ex = block_excl_scan<int64_t>(sum, &tot);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = 4 * threadIdx.x + u;
      if (k < K) s_off[k] = ex;
      ex += v[u];
    }
    if (threadIdx.x == 0) s_off[K] = tot;
  }
  __syncthreads();
  if (blockIdx.x == 0)
    for (int k = threadIdx.x; k <= K; k += kBlock) {
      pair_off[k] = s_off[k];
      if (SELF && k < K) totals[k] = s_tot[k];
    }
  __syncthreads();
  // this block's start inside every R_i, and its waves' packed prefixes
  for (int k = threadIdx.x; k < K; k += kBlock) {
    const int64_t q = static_cast<int64_t>(k) * nblk + blockIdx.x;
    if constexpr (SELF) {
      s_off[k] += s_base[k];
      blk_base[q] = s_base[k];
    } else {
      s_off[k] += blk_base[q];
    }
    s_wp[k] = wpre[q];
  }
  __syncthreads();
  const int64_t n_rows = hdr->n_out;
  const bool valid = p < n_rows;
  const int32_t y = valid ? y0 : 0;
  const int wave = threadIdx.x / kWave;
#pragma unroll
  for (int i = 0; i < kCompactPre; ++i) {
    const int32_t row = valid && i < K ? pre[i] : -1;
    const uint64_t m = __ballot(row >= 0);
    if (row >= 0) {
      const int64_t pos = s_off[i] + wave_prefix(s_wp[i], wave) + prefix_popc(m);
      pairs[pos] = make_int2(row, y);
    }
  }
  constexpr int U = 4;                  // gather-map loads in flight
  for (int i0 = kCompactPre; i0 < K; i0 += U) {
    int32_t row[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      row[u] = (valid && i0 + u < K) ? gmap[(i0 + u) * gstride + p] - 1 : -1;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u;
      const uint64_t m = __ballot(row[u] >= 0);
      if (row[u] >= 0) {
        const int64_t pos = s_off[i] + wave_prefix(s_wp[i], wave) + prefix_popc(m);
        pairs[pos] = make_int2(row[u], y);
      }
    }
  }
}

// Cell of site (b, c_1..c_d) = b << B | Z(c), where Z interleaves the bits of
// the spatial coordinates, most significant level first and coordinate 1
// first inside a level, keeping only the bits a coordinate can have
// (B = sum_j bits_j).  Walking cells in increasing order is the Z-order of
// the sites.  M[j] marks the bits of Z that hold coordinate j.
struct GridGeom {
  int D;
  int B;
  uint32_t M[kMaxD];
  int32_t size[kMaxD];
};

// Scatter bits of v into the set positions of m, lowest first.
__host__ __device__ inline uint32_t deposit(uint32_t v, uint32_t m) {
  uint32_t r = 0;
  for (uint32_t bb = 1; m; bb <<= 1) {
    const uint32_t low = m & (0u - m);
    if (v & bb) r |= low;
    m &= m - 1;
  }
  return r;
}

__device__ __forceinline__ uint32_t grid_cell(const GridGeom& g, const int32_t* x) {
  uint32_t cell = static_cast<uint32_t>(x[0]) << g.B;
  for (int j = 1; j < g.D; ++j) cell |= deposit(static_cast<uint32_t>(x[j]), g.M[j]);
  return cell;
}

// Output grid an SC emission fills as well (grid = NULL: none): grid[cell] =
// 1 + row, and with bitmap set the cell's occupancy bit too (for the
// one-launch schedule of small grids).
struct OutGrid {
  GridGeom g;
  uint32_t* grid;
  uint32_t* bitmap;
};

// SC: mark every output site some input feeds.  Output site y with
// y_j = (x_j - o_j) / s_j when that is a non-negative integer inside the
// output extent E_j; bit L(y) = lexicographic linear index of y.
__global__ __launch_bounds__(kBlock) void k_sc_mark(
    const uint64_t* __restrict__ keys, int64_t N, const int64_t* __restrict__ count, Codec cin,
    OffsetTable ot, Extents E, uint32_t* __restrict__ bitmap) {
  __shared__ int16_t s_off[kMaxK][kMaxD];
  fill_offsets(ot, s_off);
  __syncthreads();
  const int64_t r = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (r >= N || (count && r >= *count)) return;
  const uint64_t key = keys[r];
  if (key == kEmpty) return;
  int32_t x[kMaxD];
  unpack_site(cin, key, x);
  // Offsets are tried in turn even where f = s leaves one candidate: the
  // inputs of one output site then set its bit in different rounds, and all
  // but the first find it set and skip the atomic (computing the one output
  // directly and setting every lane's bit at once measured ~45 % slower).
  for (int i = 0; i < ot.K; ++i) {
    uint32_t L = 0;
    bool ok = true;
    for (int j = 0; j < ot.D; ++j) {
      const int32_t t = x[j] - s_off[i][j];
      const int32_t q = t / ot.s[j];
      ok = ok && t >= 0 && q * ot.s[j] == t && q < E.e[j];
      L = L * static_cast<uint32_t>(E.e[j]) + static_cast<uint32_t>(q);
    }
    if (ok) {
      const uint32_t bit = 1u << (L & 31);
      if (!(bitmap[L >> 5] & bit)) atomicOr(&bitmap[L >> 5], bit);
    }
  }
}

// SC on dense grids, first step in one pass over the input rows: row r is
// placed at its cell of the input grid by compare-and-swap from 0 (a cell
// found taken is a duplicate site), and the output sites it feeds are marked
// as k_sc_mark does.  With `count` set only the first *count rows exist
// (count_copy, when set, receives that count).
__global__ __launch_bounds__(kBlock) void k_sc_scatter_mark(
    const int32_t* __restrict__ coords, int64_t N, const int64_t* __restrict__ count,
    GridGeom g, uint32_t* __restrict__ grid, uint32_t* __restrict__ status,
    int64_t* __restrict__ count_copy, OffsetTable ot, Extents E, uint32_t* __restrict__ bitmap) {
  __shared__ int16_t s_off[kMaxK][kMaxD];
  fill_offsets(ot, s_off);
  __syncthreads();
  const int64_t r = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (count_copy && r == 0) *count_copy = *count;
  if (r >= N || (count && r >= *count)) return;
  int32_t x[kMaxD];
  bool ok = true;
  for (int j = 0; j < g.D; ++j) {
    x[j] = coords[r * g.D + j];
    ok = ok && x[j] >= 0 && x[j] < g.size[j];
  }
  if (!ok) {
    atomicOr(status, kStRange);
    return;
  }
  const uint32_t prev = atomicCAS(&grid[grid_cell(g, x)], 0u, static_cast<uint32_t>(r + 1));
  // (the compare-and-swap's answer is awaited only after the marking)
  for (int i = 0; i < ot.K; ++i) {
    uint32_t L = 0;
    bool in = true;
    for (int j = 0; j < ot.D; ++j) {
      const int32_t t = x[j] - s_off[i][j];
      const int32_t q = t / ot.s[j];
      in = in && t >= 0 && q * ot.s[j] == t && q < E.e[j];
      L = L * static_cast<uint32_t>(E.e[j]) + static_cast<uint32_t>(q);
    }
    if (in) {
      const uint32_t bit = 1u << (L & 31);
      if (!(bitmap[L >> 5] & bit)) atomicOr(&bitmap[L >> 5], bit);
    }
  }
  if (prev != 0u) atomicOr(status, kStDup);
}

// Popcount of 256 bitmap words per block (one word per thread).
__global__ __launch_bounds__(kBlock) void k_bitsum(const uint32_t* __restrict__ bitmap,
                                                   uint64_t nwords, uint32_t* __restrict__ bsum) {
  const uint64_t w = blockIdx.x * static_cast<uint64_t>(kBlock) + threadIdx.x;
  uint32_t tot;
  block_excl_scan<uint32_t>(w < nwords ? __popc(bitmap[w]) : 0u, &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// Single block: exclusive scan of the block sums; n_out = total.  A total
// other than `expect` (when >= 0), or than *expect_dev (when given), flags
// duplicate sites.
__global__ __launch_bounds__(kBlock) void k_bitscan(uint32_t* __restrict__ bsum, int64_t nb,
                                                    DeviceHeader* __restrict__ hdr,
                                                    int64_t expect,
                                                    const int64_t* __restrict__ expect_dev) {
  constexpr int PER = 16;                          // all requested at once
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += PER * kBlock) {
    uint32_t v[PER];
    int64_t sum = 0;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t k = base + PER * threadIdx.x + u;
      v[u] = k < nb ? bsum[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) sum += v[u];
    int64_t tot;
    int64_t ex = block_excl_scan<int64_t>(sum, &tot) + carry;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int64_t k = base + PER * threadIdx.x + u;
      if (k < nb) bsum[k] = static_cast<uint32_t>(ex);
      ex += v[u];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    hdr->n_out = carry;
    if ((expect >= 0 && carry != expect) || (expect_dev && carry != *expect_dev))
      atomicOr(&hdr->status, kStDup);
  }
}

// Emit the marked output sites in rank order: coordinates and packed keys.
// Block b works on bitmap block b / kEmitParts (256 words, whose rank base is
// bbase[b / kEmitParts]) and, of it, the 32 words of part b % kEmitParts;
// kEmitParts threads share a word, 32 / kEmitParts cells each, so a dense
// word is not emitted by one thread in 32 serial steps.  bbase = NULL (at
// most kSelfWords words): every block counts the words before its bitmap
// block itself, and the last bitmap block sets n_out, in place of k_bitsum
// and k_bitscan.
constexpr int kEmitParts = 8;
constexpr int kEmitBits = 32 / kEmitParts;
constexpr int kSelfWords = 8192;   // most words of a bitmap ranked without a scan launch
__global__ __launch_bounds__(kBlock) void k_sc_emit(
    const uint32_t* __restrict__ bitmap, uint64_t nwords, const uint32_t* __restrict__ bbase,
    Codec cout, Extents E, int32_t* __restrict__ out_coords,
    uint64_t* __restrict__ out_keys, OutGrid og, DeviceHeader* __restrict__ hdr) {
  __shared__ uint32_t s_pre[kBlock];
  __shared__ uint32_t s_word[kBlock];
  const uint64_t bw = blockIdx.x / kEmitParts;
  const int part = blockIdx.x % kEmitParts;
  uint32_t bbw = 0;                                // rank base of the bitmap block
  if (!bbase) {
    constexpr int PER = kSelfWords / kBlock;
    const uint32_t w0 = static_cast<uint32_t>(bw) * kBlock;
    uint32_t v[PER], before = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {                // every load in flight at once
      const uint32_t idx = k * kBlock + threadIdx.x;
      v[k] = bitmap[idx < w0 ? idx : 0u];
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) before += k * kBlock + threadIdx.x < w0 ? __popc(v[k]) : 0u;
    block_excl_scan<uint32_t>(before, &bbw);
  } else {
    bbw = bbase[bw];
  }
  {
    // exclusive popcount prefix over the 256 words of the bitmap block
    const uint64_t w = bw * kBlock + threadIdx.x;
    const uint32_t tw = w < nwords ? bitmap[w] : 0u;
    uint32_t tot;
    s_word[threadIdx.x] = tw;
    s_pre[threadIdx.x] = block_excl_scan<uint32_t>(__popc(tw), &tot);
    if (!bbase && blockIdx.x == gridDim.x - kEmitParts && threadIdx.x == 0)
      hdr->n_out = static_cast<int64_t>(bbw) + tot;
  }
  __syncthreads();
  const int wi = part * (kBlock / kEmitParts) + threadIdx.x / kEmitParts;   // word in block
  const int sub = threadIdx.x % kEmitParts;
  const uint64_t w = bw * kBlock + wi;
  if (w >= nwords) return;
  const uint32_t full = s_word[wi];
  const uint32_t below = (1u << (sub * kEmitBits)) - 1u;
  uint32_t word = (full >> (sub * kEmitBits)) & ((1u << kEmitBits) - 1u);
  if (!word) return;
  uint32_t rank = bbw + s_pre[wi] + __popc(full & below);
  // coordinates of the thread's first cell (one division per dimension); a
  // set bit b adds b to the last coordinate, carried into the others only
  // when it passes the extent
  int32_t y0[kMaxD];
  {
    uint32_t L = static_cast<uint32_t>(w * 32 + sub * kEmitBits);
    for (int j = cout.D - 1; j >= 0; --j) {
      y0[j] = static_cast<int32_t>(L % static_cast<uint32_t>(E.e[j]));
      L /= static_cast<uint32_t>(E.e[j]);
    }
  }
  while (word) {
    const int b = __builtin_ctz(word);
    word &= word - 1;
    int32_t yv[kMaxD];
    for (int j = 0; j < cout.D; ++j) yv[j] = y0[j];
    yv[cout.D - 1] += b;
    for (int j = cout.D - 1; j > 0 && yv[j] >= E.e[j]; --j) {
      yv[j - 1] += yv[j] / E.e[j];
      yv[j] %= E.e[j];
    }
    if (cout.D == 4) {
      reinterpret_cast<int4*>(out_coords)[rank] = make_int4(yv[0], yv[1], yv[2], yv[3]);
    } else {
      for (int j = 0; j < cout.D; ++j) out_coords[static_cast<int64_t>(rank) * cout.D + j] = yv[j];
    }
    if (out_keys) out_keys[rank] = pack_site(cout, yv);
    if (og.grid) {
      const uint32_t cell = grid_cell(og.g, yv);
      og.grid[cell] = rank + 1;
      if (og.bitmap) atomicOr(&og.bitmap[cell >> 5], 1u << (cell & 31));
    }
    ++rank;
  }
}

// Forward schedule: Morton code of every output row (sample index on top,
// then the spatial coordinates' bits interleaved from the most significant),
// sorted together with the row index.  Consecutive rows of the sorted order
// are spatially compact, so a tile of them touches a small halo of inputs.
template <int D>
__global__ __launch_bounds__(kBlock) void k_morton(const uint64_t* __restrict__ rowkeys,
                                                   const DeviceHeader* __restrict__ hdr,
                                                   Codec c, int maxb, int sbits,
                                                   uint64_t* __restrict__ mk,
                                                   int32_t* __restrict__ mv) {
  const int64_t y = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (y >= hdr->n_out) return;
  const uint64_t key = rowkeys[y];
  uint32_t v[D];
#pragma unroll
  for (int j = 0; j < D; ++j) v[j] = static_cast<uint32_t>((key >> c.shift[j]) & c.fmask[j]);
  uint64_t m = 0;
  for (int L = maxb - 1; L >= 0; --L) {
#pragma unroll
    for (int j = 1; j < D; ++j)
      if (c.fmask[j] >> L) m = (m << 1) | ((v[j] >> L) & 1u);
  }
  m |= static_cast<uint64_t>(v[0]) << sbits;
  mk[y] = m;
  mv[y] = static_cast<int32_t>(y);
}

// The sorted-brick build's first pass over the sites: packed key of row r (kEmpty: out of range, flagged), the
// coordinates copied, and the Morton code of the key with r beside it.
template <int D>
__global__ __launch_bounds__(kBlock) void k_site_morton(
    const int32_t* __restrict__ coords, int64_t N, Codec c, uint64_t* __restrict__ keys,
    int32_t* __restrict__ copy_out, uint32_t* __restrict__ status, int maxb, int sbits,
    uint64_t* __restrict__ mk, int32_t* __restrict__ mv) {
  const int64_t r = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (r >= N) return;
  int32_t x[D];
  bool ok = true;
#pragma unroll
  for (int j = 0; j < D; ++j) {
    x[j] = coords[r * D + j];
    ok = ok && x[j] >= 0 && x[j] < c.size[j];
    if (copy_out) copy_out[r * D + j] = x[j];
  }
  const uint64_t key = ok ? pack_site(c, x) : kEmpty;
  keys[r] = key;
  if (!ok) atomicOr(status, kStRange);
  uint32_t v[D];
#pragma unroll
  for (int j = 0; j < D; ++j) v[j] = static_cast<uint32_t>((key >> c.shift[j]) & c.fmask[j]);
  uint64_t m = 0;
  for (int L = maxb - 1; L >= 0; --L) {
#pragma unroll
    for (int j = 1; j < D; ++j)
      if (c.fmask[j] >> L) m = (m << 1) | ((v[j] >> L) & 1u);
  }
  m |= static_cast<uint64_t>(v[0]) << sbits;
  mk[r] = m;
  mv[r] = static_cast<int32_t>(r);
}

// ---------------------------------------------------------------------------
// Dense index grid (used when the grid is small enough to hold one int32 per
// cell; the sites' cells are laid out along the Z-order curve)
// ---------------------------------------------------------------------------
// Place input row r at its cell: grid[cell] = r + 1 (0 = empty).  With CAS,
// by compare-and-swap from 0, and a cell found taken is a duplicate site.
// Without it a plain store; duplicates then leave fewer occupied cells than
// rows, which the schedule's count reveals (k_bitscan's `expect`).
// Optionally copies the coordinates (VSC output sites) and writes packed
// keys (SC marking).  With `count` set, only the first *count (<= N) rows
// exist.
// With `bitmap` set, the cell's occupancy bit is set too (the bitmap cleared
// with the grid), for the one-launch schedule of small grids.
template <bool CAS>
__global__ __launch_bounds__(kBlock) void k_grid_scatter(
    const int32_t* __restrict__ coords, int64_t N, const int64_t* __restrict__ count,
    GridGeom g, uint32_t* __restrict__ grid, int32_t* __restrict__ copy_out, Codec ckey,
    uint64_t* __restrict__ keys_out, uint32_t* __restrict__ status,
    int64_t* __restrict__ count_copy, uint32_t* __restrict__ bitmap) {
  const int64_t r = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
  if (count_copy && r == 0) *count_copy = *count;   // the book's own copy of the row count
  if (r >= N || (count && r >= *count)) return;
  int32_t x[kMaxD];
  bool ok = true;
  for (int j = 0; j < g.D; ++j) {
    x[j] = coords[r * g.D + j];
    ok = ok && x[j] >= 0 && x[j] < g.size[j];
    if (copy_out) copy_out[r * g.D + j] = x[j];
  }
  if (!ok) {
    if (keys_out) keys_out[r] = kEmpty;
    atomicOr(status, kStRange);
    return;
  }
  if (keys_out) keys_out[r] = pack_site(ckey, x);
  const uint32_t cell = grid_cell(g, x);
  if (bitmap) atomicOr(&bitmap[cell >> 5], 1u << (cell & 31));
  if (!CAS)
    grid[cell] = static_cast<uint32_t>(r + 1);
  else if (atomicCAS(&grid[cell], 0u, static_cast<uint32_t>(r + 1)) != 0u)
    atomicOr(status, kStDup);
}

// Occupancy bitmap of the grid, one word (32 cells) per thread, and the
// number of occupied cells of every block of 256 words.
__global__ __launch_bounds__(kBlock) void k_grid_bits(const uint32_t* __restrict__ grid,
                                                      uint64_t cells, uint64_t nwords,
                                                      uint32_t* __restrict__ bitmap,
                                                      uint32_t* __restrict__ bsum) {
  const uint64_t w = blockIdx.x * static_cast<uint64_t>(kBlock) + threadIdx.x;
  uint32_t word = 0;
  if (w < nwords) {
    if (32 * w + 32 <= cells) {
      const uint4* q = reinterpret_cast<const uint4*>(grid + 32 * w);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint4 v = q[k];
        word |= (v.x ? 1u : 0u) << (4 * k) | (v.y ? 2u : 0u) << (4 * k) |
                (v.z ? 4u : 0u) << (4 * k) | (v.w ? 8u : 0u) << (4 * k);
      }
    } else {
      for (uint64_t c = 32 * w; c < cells; ++c)
        word |= (grid[c] ? 1u : 0u) << (c - 32 * w);
    }
    bitmap[w] = word;
  }
  uint32_t tot;
  block_excl_scan<uint32_t>(__popc(word), &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// Rows of the occupied cells in cell order -> perm (the Z-order schedule),
// one bitmap word per thread; block bases from k_grid_bits + k_bitscan.
// SELF (at most kSelfBlocks blocks): bbase holds k_grid_bits' block sums as
// they are; every block adds up those before its own (a few loads per
// thread), and the last block sets n_out to the occupied cells and flags
// duplicate sites as k_bitscan would (a count other than `expect` when >= 0,
// or than *expect_dev when given).
constexpr int kSelfBlocks = 4096;
template <bool SELF>
__global__ __launch_bounds__(kBlock) void k_grid_emit(const uint32_t* __restrict__ bitmap,
                                                      uint64_t nwords, uint64_t cells,
                                                      const uint32_t* __restrict__ bbase,
                                                      const uint32_t* __restrict__ grid,
                                                      int32_t* __restrict__ perm,
                                                      DeviceHeader* __restrict__ hdr,
                                                      int64_t expect,
                                                      const int64_t* __restrict__ expect_dev) {
  const uint64_t w = blockIdx.x * static_cast<uint64_t>(kBlock) + threadIdx.x;
  const uint32_t word = w < nwords ? bitmap[w] : 0u;
  uint32_t base;
  if constexpr (SELF) {
    constexpr int PER = kSelfBlocks / kBlock;
    uint32_t v[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {                // every load in flight at once
      const uint32_t idx = k * kBlock + threadIdx.x;
      v[k] = idx < blockIdx.x ? bbase[idx] : 0u;
    }
    uint32_t before = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) before += v[k];
    block_excl_scan<uint32_t>(before, &base);
  } else {
    base = bbase[blockIdx.x];
  }
  uint32_t tot;
  uint32_t rank = block_excl_scan<uint32_t>(__popc(word), &tot) + base;
  if (SELF && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    const int64_t t = static_cast<int64_t>(base) + tot;
    if ((expect >= 0 && t != expect) || (expect_dev && t != *expect_dev))
      atomicOr(&hdr->status, kStDup);
    hdr->n_out = t;
  }
  if (!word) return;
  // the word's 32 cells as eight 16-byte loads issued together (a loop of
  // one load per occupied cell waits out each load's latency in turn); a
  // word's cells are whole 16-byte groups except in a grid's last word,
  // where the cells past the end are not read
  uint32_t v[32];
  if (32 * w + 32 <= cells) {
    const uint4* q = reinterpret_cast<const uint4*>(grid + 32 * w);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint4 t = q[k];
      v[4 * k] = t.x;
      v[4 * k + 1] = t.y;
      v[4 * k + 2] = t.z;
      v[4 * k + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 32; ++k) v[k] = 32 * w + k < cells ? grid[32 * w + k] : 0u;
  }
#pragma unroll
  for (int k = 0; k < 32; ++k)
    if ((word >> k) & 1u) perm[rank++] = static_cast<int32_t>(v[k]) - 1;
}

// Small grids (at most kSelfWords bitmap words, the bitmap set by the
// scatter): the schedule in one launch instead of three.  Blocks are laid
// out as in k_sc_emit (bitmap block b / kEmitParts, its words' part b %
// kEmitParts, kEmitParts threads per word); every block finds its bitmap
// block's base itself, as the popcount of all the words before it (at most
// kSelfWords words, loaded by all its threads at once), and each thread
// emits the rows of its 4 cells (one 16-byte grid load).  The last bitmap
// block sets n_out to the occupied cells; a count other than `expect` (when
// >= 0), or than *expect_dev (when given), flags duplicate sites.
__global__ __launch_bounds__(kBlock) void k_grid_emit_self(
    const uint32_t* __restrict__ bitmap, uint64_t nwords, uint64_t cells,
    const uint32_t* __restrict__ grid, int32_t* __restrict__ perm,
    DeviceHeader* __restrict__ hdr, int64_t expect, const int64_t* __restrict__ expect_dev) {
  constexpr int PER = kSelfWords / kBlock;
  static_assert(kEmitBits == 4, "a thread's cells are one 16-byte group of the grid");
  __shared__ uint32_t s_pre[kBlock];
  __shared__ uint32_t s_word[kBlock];
  const uint32_t bw = blockIdx.x / kEmitParts;
  const int part = blockIdx.x % kEmitParts;
  const uint32_t w0 = bw * kBlock;                 // first word of the bitmap block
  uint32_t v[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {                  // every load in flight at once
    const uint32_t idx = k * kBlock + threadIdx.x;
    v[k] = bitmap[idx < w0 ? idx : 0u];
  }
  const uint64_t wt = w0 + threadIdx.x;
  const uint32_t tword = wt < nwords ? bitmap[wt] : 0u;
  uint32_t before = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) before += k * kBlock + threadIdx.x < w0 ? __popc(v[k]) : 0u;
  uint32_t base, tot;
  block_excl_scan<uint32_t>(before, &base);
  s_word[threadIdx.x] = tword;
  s_pre[threadIdx.x] = block_excl_scan<uint32_t>(__popc(tword), &tot);
  if (blockIdx.x == gridDim.x - kEmitParts && threadIdx.x == 0) {
    const int64_t t = static_cast<int64_t>(base) + tot;
    if ((expect >= 0 && t != expect) || (expect_dev && t != *expect_dev))
      atomicOr(&hdr->status, kStDup);
    hdr->n_out = t;
  }
  __syncthreads();
  const int wi = part * (kBlock / kEmitParts) + threadIdx.x / kEmitParts;   // word in block
  const int sub = threadIdx.x % kEmitParts;
  const uint64_t w = w0 + wi;
  if (w >= nwords) return;
  const uint32_t full = s_word[wi];
  const uint32_t bits = (full >> (sub * kEmitBits)) & ((1u << kEmitBits) - 1u);
  if (!bits) return;
  uint32_t rank = base + s_pre[wi] + __popc(full & ((1u << (sub * kEmitBits)) - 1u));
  const uint64_t c0 = 32 * w + sub * kEmitBits;
  uint32_t c[kEmitBits];
  if (c0 + kEmitBits <= cells) {
    const uint4 t = *reinterpret_cast<const uint4*>(grid + c0);
    c[0] = t.x;
    c[1] = t.y;
    c[2] = t.z;
    c[3] = t.w;
  } else {
#pragma unroll
    for (int k = 0; k < kEmitBits; ++k) c[k] = c0 + k < cells ? grid[c0 + k] : 0u;
  }
#pragma unroll
  for (int k = 0; k < kEmitBits; ++k)
    if ((bits >> k) & 1u) perm[rank++] = static_cast<int32_t>(c[k]) - 1;
}

typedef uint32_t dw4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kBufDword3 = 0x00020000u;   // gfx9 raw buffer descriptor word 3
constexpr uint32_t kOOB = 0x80000000u;         // byte offset past every buffer: loads 0

// Neighbour probe on the dense grid.  Thread = schedule position p, output
// row y = perm[p] with site c (rows_sites[y]).  The input site of offset i
// is c + o_i - r (VSC) or s*c + o_i (SC); its cell follows from c's cell by
// one dilated addition per dimension, ((Z_j | ~M_j) + Z(o_ij)) & M_j, which
// carries through the bits of the other dimensions.  The grid holds 1 + row
// (0 = empty), which is the gather-map entry as it stands.  Every lookup of
// a batch is an unconditional buffer load (off-grid neighbours use an offset
// past the buffer, which reads 0), so the whole batch is in flight at once.
template <bool SC, int D>
__global__ __launch_bounds__(kBlock) void k_probe_grid(
    const int32_t* __restrict__ rows_sites, const int32_t* __restrict__ perm,
    const DeviceHeader* __restrict__ hdr, int64_t gstride, GridGeom g, OffsetTable ot,
    const uint32_t* __restrict__ grid, uint32_t cells, int32_t* __restrict__ gmap,
    int32_t* __restrict__ blk_cnt, uint32_t* __restrict__ wpre, int64_t nblk) {
  const int64_t blk = probe_block(hdr->n_out, nblk);
  if (blk < 0) return;
  __shared__ int16_t s_off[kMaxK][kMaxD];
  __shared__ uint32_t s_dil[kMaxK][kMaxD];
  __shared__ uint8_t s_cnt[kMaxK][kBlock / kWave];
  for (int i = threadIdx.x; i < ot.K; i += blockDim.x) {
    int rem = i;
    for (int j = ot.D - 1; j >= 0; --j) {
      const int o = rem % ot.f[j] - ot.r[j];
      rem /= ot.f[j];
      s_off[i][j] = static_cast<int16_t>(o);
      const uint32_t low = (1u << __popc(g.M[j])) - 1u;
      s_dil[i][j] = j ? deposit(static_cast<uint32_t>(o) & low, g.M[j]) : 0u;
    }
  }
  __syncthreads();

  const int64_t n_rows = hdr->n_out;
  const int64_t p = blk * kBlock + threadIdx.x;
  const bool valid = p < n_rows;
  const int wave = threadIdx.x / kWave;
  const int32_t y = valid ? perm[p] : 0;
  int32_t c[D];
  uint32_t zc[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    c[j] = valid ? rows_sites[static_cast<int64_t>(y) * D + j] : 0;
    if (SC) c[j] *= ot.s[j];
    zc[j] = j ? (deposit(static_cast<uint32_t>(c[j]), g.M[j]) | ~g.M[j]) : 0u;
  }
  const uint32_t base = static_cast<uint32_t>(c[0]) << g.B;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(grid), 0, static_cast<int>(cells * 4), static_cast<int>(kBufDword3));

  constexpr int NB = 14;
  for (int i0 = 0; i0 < ot.K; i0 += NB) {
    uint32_t gv[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int i = i0 + u;
      const int ic = i < ot.K ? i : ot.K - 1;
      bool ok = valid && i < ot.K && i != ot.centre;
      uint32_t cell = base;
#pragma unroll
      for (int j = 1; j < D; ++j) {
        const int32_t n = c[j] + s_off[ic][j];
        ok = ok && n >= 0 && n < g.size[j];
        cell |= (zc[j] + s_dil[ic][j]) & g.M[j];
      }
      gv[u] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, ok ? cell * 4 : kOOB, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int i = i0 + u;
      if (i >= ot.K) break;
      const int32_t e = (valid && i == ot.centre) ? y + 1 : static_cast<int32_t>(gv[u]);
      if (p < gstride) gmap[i * gstride + p] = e;   // 1 + input row, 0 = none
      const uint64_t m = __ballot(e != 0);
      if (lane_id() == 0) s_cnt[i][wave] = static_cast<uint8_t>(__popcll(m));
    }
  }
  publish_counts(s_cnt, ot.K, blk_cnt, wpre, nblk, blk);
}

// The same probe for VSC 3x3x3 on a 4-D grid (sample + 3 coordinates) whose
// two lowest Z bits are the lowest bits of coordinates 3 and 2: the four
// cells that differ only there are 16 contiguous bytes, so the 3 x 3 window
// of a cell in those coordinates lies in 2 x 2 such groups, and 12 16-byte
// loads cover the 26 neighbours where the generic probe makes 26 4-byte
// loads (each of which costs the L1 a tag lookup per lane).  Group addresses
// stay inside the grid even for neighbours off its edge (the dilated
// addition wraps within the coordinate's bits); those are masked by the
// coordinate range checks.  Offset i = 9 (dx + 1) + 3 (dy + 1) + (dz + 1).
//
// It runs twice.  WRITE = false counts, per block and offset, the positions
// with a neighbour (and the per-wave prefixes), which k_scan turns into each
// block's base inside every R_i; it needs occupancy only, so it reads the
// same four-cell groups from the occupancy bitmap (4 bits of a word, 1/32 of
// the grid's bytes) instead of the grid.  WRITE = true repeats the lookups in
// the grid and writes the gather map and, at once, every pair at its final
// place in R_i (pair_off[i] + the block's base + the waves before it + the
// set lanes before it), so the pair lists never need a second pass over the
// gather map.  Workgroup 0 of the writing pass also stores pair_off.
template <bool WRITE>
__global__ __launch_bounds__(kBlock) void k_probe_grid_g4(
    const int32_t* __restrict__ rows_sites, const int32_t* __restrict__ perm,
    const DeviceHeader* __restrict__ hdr, int64_t gstride, GridGeom g,
    const uint32_t* __restrict__ grid, uint32_t cells, const uint32_t* __restrict__ bitmap,
    int32_t* __restrict__ gmap, int32_t* __restrict__ blk_cnt, uint32_t* __restrict__ wpre,
    int64_t nblk, const int64_t* __restrict__ totals, int2* __restrict__ pairs,
    int64_t* __restrict__ pair_off) {
  __shared__ uint8_t s_cnt[kMaxK][kBlock / kWave];
  __shared__ int64_t s_off[28];
  __shared__ uint32_t s_wp[27];
  if constexpr (WRITE) {
    // pair_off = exclusive prefix of the 27 totals
    if (threadIdx.x < kWave) {
      const int64_t t = threadIdx.x < 27 ? totals[threadIdx.x] : 0;
      const int64_t inc = wave_incl_scan(t);
      if (threadIdx.x < 28) s_off[threadIdx.x] = inc - t;
    }
    __syncthreads();
    if (blockIdx.x == 0 && threadIdx.x < 28) pair_off[threadIdx.x] = s_off[threadIdx.x];
  }
  const int64_t blk = probe_block(hdr->n_out, nblk);
  if (blk < 0) return;
  if constexpr (WRITE) {
    if (threadIdx.x < 27) {
      const int64_t q = static_cast<int64_t>(threadIdx.x) * nblk + blk;
      s_off[threadIdx.x] += blk_cnt[q];
      s_wp[threadIdx.x] = wpre[q];
    }
    __syncthreads();
  }
  const int64_t n_rows = hdr->n_out;
  const int64_t p = blk * kBlock + threadIdx.x;
  const bool valid = p < n_rows;
  const int wave = threadIdx.x / kWave;
  const int32_t y = valid ? perm[p] : 0;
  int4 c = make_int4(0, 0, 0, 0);
  if (valid) c = reinterpret_cast<const int4*>(rows_sites)[y];
  // dilated +1 / -1 in every coordinate (uniform)
  // (-1 in a coordinate's bits is all of them; +1 is the lowest)
  uint32_t dp[4], dm[4];
#pragma unroll
  for (int j = 1; j < 4; ++j) {
    dm[j] = g.M[j];
    dp[j] = g.M[j] & (0u - g.M[j]);
  }
  const uint32_t z1 = deposit(static_cast<uint32_t>(c.y), g.M[1]) | ~g.M[1];
  const uint32_t z2 = deposit(static_cast<uint32_t>(c.z), g.M[2]) | ~g.M[2];
  const uint32_t z3 = deposit(static_cast<uint32_t>(c.w), g.M[3]) | ~g.M[3];
  const uint32_t base = static_cast<uint32_t>(c.x) << g.B;
  const uint32_t xp[3] = {(z1 + dm[1]) & g.M[1], z1 & g.M[1], (z1 + dp[1]) & g.M[1]};
  const uint32_t yp[2] = {(z2 + dm[2]) & g.M[2], (z2 + dp[2]) & g.M[2]};
  const uint32_t zp[2] = {(z3 + dm[3]) & g.M[3], (z3 + dp[3]) & g.M[3]};
  dw4 v[3][2][2];          // WRITE: the groups' four cells
  uint32_t nib[3][2][2];   // otherwise: their four occupancy bits
  if constexpr (WRITE) {
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(grid), 0, static_cast<int>(cells * 4),
        static_cast<int>(kBufDword3));
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          const uint32_t cell = (base | xp[a] | yp[b] | zp[d]) & ~3u;
          v[a][b][d] = __builtin_bit_cast(
              dw4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, valid ? cell * 4 : kOOB, 0, 0));
        }
  } else {
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(bitmap), 0, static_cast<int>(((cells + 31) / 32) * 4),
        static_cast<int>(kBufDword3));
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          const uint32_t cell = (base | xp[a] | yp[b] | zp[d]) & ~3u;
          const uint32_t word =
              __builtin_amdgcn_raw_buffer_load_b32(rsrc, valid ? (cell >> 5) * 4 : kOOB, 0, 0);
          nib[a][b][d] = (word >> (cell & 31u)) & 15u;
        }
  }
  const int yo = c.z & 1, zo = c.w & 1;
  bool xok[3], yok[3], zok[3];
#pragma unroll
  for (int o = 0; o < 3; ++o) {
    xok[o] = valid && c.y + o - 1 >= 0 && c.y + o - 1 < g.size[1];
    yok[o] = c.z + o - 1 >= 0 && c.z + o - 1 < g.size[2];
    zok[o] = c.w + o - 1 >= 0 && c.w + o - 1 < g.size[3];
  }
#pragma unroll
  for (int i = 0; i < 27; ++i) {
    const int dx = i / 9, dy = (i / 3) % 3, dz = i % 3;   // 0, 1, 2 = -1, 0, +1
    int32_t e;
    if (i == 13) {
      e = valid ? y + 1 : 0;
    } else {
      // group in y: the lower one holds y - 1 (and y when y is odd)
      const bool bh = dy == 2 || (dy == 1 && !yo);
      const bool dh = dz == 2 || (dz == 1 && !zo);
      const int ey = dy == 1 ? yo : yo ^ 1;       // bit 0 of y + dy - 1
      const int ez = dz == 1 ? zo : zo ^ 1;
      uint32_t val;
      if constexpr (WRITE) {
        const dw4 w0 = bh ? v[dx][1][0] : v[dx][0][0];
        const dw4 w1 = bh ? v[dx][1][1] : v[dx][0][1];
        const dw4 w = dh ? w1 : w0;
        const uint32_t lo = ez ? w.y : w.x, hi = ez ? w.w : w.z;
        val = ey ? hi : lo;
      } else {
        // cell 2 ey + ez of the group (bit 0: coordinate 3, bit 1: coordinate 2)
        const uint32_t n0 = bh ? nib[dx][1][0] : nib[dx][0][0];
        const uint32_t n1 = bh ? nib[dx][1][1] : nib[dx][0][1];
        val = ((dh ? n1 : n0) >> (2 * ey + ez)) & 1u;
      }
      e = (xok[dx] && yok[dy] && zok[dz]) ? static_cast<int32_t>(val) : 0;
    }
    const uint64_t m = __ballot(e != 0);
    if constexpr (WRITE) {
      if (p < gstride) gmap[i * gstride + p] = e;   // 1 + input row, 0 = none
      if (e != 0)
        pairs[s_off[i] + wave_prefix(s_wp[i], wave) + prefix_popc(m)] = make_int2(e - 1, y);
    } else {
      if (lane_id() == 0) s_cnt[i][wave] = static_cast<uint8_t>(__popcll(m));
    }
  }
  if constexpr (!WRITE) publish_counts(s_cnt, 27, blk_cnt, wpre, nblk, blk);
}

// SC 2^3 with stride 2 on a 4-D grid whose three lowest Z bits are the lowest
// bits of coordinates 3, 2, 1: the receptive field of output site c is the
// aligned 2 x 2 x 2 cube at 2c, 8 consecutive cells (32 bytes) in the order
// of the offsets (i = 4 o_1 + 2 o_2 + o_3), read with two 16-byte loads
// instead of eight 4-byte ones.
__global__ __launch_bounds__(kBlock) void k_probe_grid_sc2(
    const int32_t* __restrict__ rows_sites, const int32_t* __restrict__ perm,
    const DeviceHeader* __restrict__ hdr, int64_t gstride, GridGeom g,
    const uint32_t* __restrict__ grid, uint32_t cells, int32_t* __restrict__ gmap,
    int32_t* __restrict__ blk_cnt, uint32_t* __restrict__ wpre, int64_t nblk) {
  const int64_t blk = probe_block(hdr->n_out, nblk);
  if (blk < 0) return;
  __shared__ uint8_t s_cnt[kMaxK][kBlock / kWave];
  const int64_t n_rows = hdr->n_out;
  const int64_t p = blk * kBlock + threadIdx.x;
  const bool valid = p < n_rows;
  const int wave = threadIdx.x / kWave;
  const int32_t y = valid ? perm[p] : 0;
  int4 c = make_int4(0, 0, 0, 0);
  if (valid) c = reinterpret_cast<const int4*>(rows_sites)[y];
  const uint32_t cell = (static_cast<uint32_t>(c.x) << g.B) |
                        deposit(2u * static_cast<uint32_t>(c.y), g.M[1]) |
                        deposit(2u * static_cast<uint32_t>(c.z), g.M[2]) |
                        deposit(2u * static_cast<uint32_t>(c.w), g.M[3]);
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(grid), 0, static_cast<int>(cells * 4), static_cast<int>(kBufDword3));
  const dw4 v0 = __builtin_bit_cast(
      dw4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, valid ? cell * 4 : kOOB, 0, 0));
  const dw4 v1 = __builtin_bit_cast(
      dw4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, valid ? cell * 4 + 16 : kOOB, 0, 0));
  const uint32_t cv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int o1 = i >> 2, o2 = (i >> 1) & 1, o3 = i & 1;
    const bool ok = valid && 2 * c.y + o1 < g.size[1] && 2 * c.z + o2 < g.size[2] &&
                    2 * c.w + o3 < g.size[3];
    const int32_t e = ok ? static_cast<int32_t>(cv[i]) : 0;
    if (p < gstride) gmap[i * gstride + p] = e;   // 1 + input row, 0 = none
    const uint64_t m = __ballot(e != 0);
    if (lane_id() == 0) s_cnt[i][wave] = static_cast<uint8_t>(__popcll(m));
  }
  publish_counts(s_cnt, 8, blk_cnt, wpre, nblk, blk);
}

// ---------------------------------------------------------------------------
// Host orchestration
// ---------------------------------------------------------------------------

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    T* p = reinterpret_cast<T*>(base + off);
    off = align_up(off + count * sizeof(T), 256);
    return p;
  }
};

inline unsigned grid_for(int64_t n, int per = kBlock) {
  int64_t g = (n + per - 1) / per;
  return static_cast<unsigned>(g < 1 ? 1 : g);
}

void launch_zero(uint32_t* p, uint64_t n, hipStream_t stream, DeviceHeader* hdr = nullptr,
                 int64_t n_out = 0) {
  const uint64_t n4 = n / 4;
  uint64_t blocks = (n4 + 4 * kBlock - 1) / (4 * kBlock);   // 4 stores per thread
  blocks = blocks < 1 ? 1 : (blocks > 65536 ? 65536 : blocks);
  k_zero_u32<<<static_cast<unsigned>(blocks), kBlock, 0, stream>>>(p, n, hdr, n_out);
}

OffsetTable make_offsets(spconv_rulebook rb) {
  OffsetTable ot{};
  ot.K = static_cast<int>(rb->K);
  ot.D = rb->D;
  int centre = 0;
  for (int j = 0; j < rb->D; ++j) {
    ot.f[j] = rb->f[j];
    ot.s[j] = rb->s[j];
    ot.r[j] = rb->kind == SPCONV_VSC ? (rb->f[j] - 1) / 2 : 0;
    centre = centre * rb->f[j] + ot.r[j];
  }
  ot.centre = rb->kind == SPCONV_VSC ? centre : -1;
  return ot;
}

// Table geometry: slots = power of two >= 4N (at least 64), so a home bucket
// of 4 is rarely full; the test-only environment variable
// SPCONV_TEST_HASH_SLOTS forces a (tiny) slot count.
uint64_t table_slots(int64_t N) {
  if (const char* e = std::getenv("SPCONV_TEST_HASH_SLOTS")) {
    uint64_t v = std::strtoull(e, nullptr, 10);
    uint64_t p = 4;
    while (p < v) p <<= 1;
    return p;
  }
  uint64_t p = 64;
  while (p < 4ull * static_cast<uint64_t>(N)) p <<= 1;
  return p;
}

struct Transient {
  void* mem = nullptr;
  uint64_t* keys = nullptr;
  Table table{};
  bool wide = false;
};

int alloc_transient(spconv_rulebook rb, int64_t N, const Codec& cin, size_t extra_bytes,
                    Transient* tr, Carver* cv) {
  const uint64_t slots = table_slots(N);
  const int rbits = bitlen(static_cast<uint64_t>(N));
  tr->wide = cin.kbits + rbits > 64;
  size_t bytes = align_up(N * sizeof(uint64_t), 256) + align_up(slots * 8, 256) +
                 (tr->wide ? align_up(slots * 4, 256) : 0) + extra_bytes + 256;
  if (dev_alloc(rb, bytes, rb->stream, &tr->mem) != SPCONV_OK) return SPCONV_ENOMEM;
  cv->base = static_cast<char*>(tr->mem);
  tr->keys = cv->take<uint64_t>(N);
  tr->table.slots = cv->take<uint64_t>(slots);
  tr->table.vals = tr->wide ? cv->take<int32_t>(slots) : nullptr;
  tr->table.nbuckets = slots / 4;
  tr->table.rbits = tr->wide ? 0 : rbits;
  // brick = the key with the lowest bit of every spatial coordinate cleared;
  // the first two spatial low bits pick the bucket inside the home line
  uint64_t low = 0;
  tr->table.lmask1 = tr->table.lmask0 = 0;
  int picked = 0;
  for (int j = 1; j < cin.D; ++j) {
    if (cin.fmask[j] == 0) continue;
    const uint64_t bit = 1ull << cin.shift[j];
    low |= bit;
    if (picked == 0) tr->table.lmask1 = bit;
    else if (picked == 1) tr->table.lmask0 = bit;
    ++picked;
  }
  tr->table.brick_mask = ~low;
  tr->table.line_shift = 2;
  if (const char* e = std::getenv("SPCONV_HASH_LAYOUT")) {
    if (std::strcmp(e, "random") == 0) {     // one bucket per line, hash of the whole key
      tr->table.brick_mask = ~0ull;
      tr->table.lmask1 = tr->table.lmask0 = 0;
      tr->table.line_shift = 0;
    }
  }
  return SPCONV_OK;
}

size_t schedule_bytes(int64_t n_cap) {
  return 2 * align_up(static_cast<size_t>(n_cap) * 8, 256) +
         2 * align_up(static_cast<size_t>(n_cap) * 4, 256) +
         align_up(radix_sort_scratch_bytes(n_cap), 256);
}

// Output rows in Morton order -> rb->perm (scratch carved from the transient
// allocation by `cv`); returns the sorted Morton codes.  With lo_bit > 0 the
// lowest lo_bit bits of the codes are left out of the sort (the brick map
// orders each brick's sites itself).  With si the site keys (si->keys, which
// is rowkeys) are packed in the same pass as the Morton codes.
struct SiteIn {
  const int32_t* coords;
  int64_t N;
  uint64_t* keys;
  int32_t* copy_out;
  uint32_t* status;
};
const uint64_t* launch_schedule(spconv_rulebook rb, const uint64_t* rowkeys, const Codec& crow,
                                Carver* cv, int lo_bit, const SiteIn* si) {
  const int64_t n = rb->n_cap;
  int maxb = 0, sbits = 0;
  for (int j = 1; j < crow.D; ++j) {
    const int b = bitlen(crow.fmask[j]);
    maxb = b > maxb ? b : maxb;
    sbits += b;
  }
  const int total = sbits + bitlen(crow.fmask[0]);
  // the values ping-pong between two arrays, one of them the schedule itself,
  // chosen so that the last pass lands in it
  const bool odd = radix_sort_passes(total, lo_bit) % 2 == 1;
  uint64_t* mk = cv->take<uint64_t>(n);
  uint64_t* mk2 = cv->take<uint64_t>(n);
  int32_t* mv = odd ? cv->take<int32_t>(n) : rb->perm;
  int32_t* mv2 = odd ? rb->perm : cv->take<int32_t>(n);
  void* scratch = cv->take<unsigned char>(radix_sort_scratch_bytes(n));
  const unsigned g = grid_for(n);
  if (si) {
    const unsigned gs = grid_for(si->N);
#define SPC_SITE_MORTON(DD)                                                                   \
  k_site_morton<DD><<<gs, kBlock, 0, rb->stream>>>(si->coords, si->N, crow, si->keys,          \
                                                   si->copy_out, si->status, maxb, sbits, mk, mv)
    switch (crow.D) {
      case 2: SPC_SITE_MORTON(2); break;
      case 3: SPC_SITE_MORTON(3); break;
      default: SPC_SITE_MORTON(4); break;
    }
#undef SPC_SITE_MORTON
  } else {
    switch (crow.D) {
      case 2: k_morton<2><<<g, kBlock, 0, rb->stream>>>(rowkeys, rb->hdr, crow, maxb, sbits, mk, mv); break;
      case 3: k_morton<3><<<g, kBlock, 0, rb->stream>>>(rowkeys, rb->hdr, crow, maxb, sbits, mk, mv); break;
      default: k_morton<4><<<g, kBlock, 0, rb->stream>>>(rowkeys, rb->hdr, crow, maxb, sbits, mk, mv); break;
    }
  }
  const bool in_tmp =
      radix_sort_pairs(mk, mv, mk2, mv2, rb->hdr, n, total, scratch, rb->stream, lo_bit);
  return in_tmp ? mk2 : mk;
}

int launch_insert(spconv_rulebook rb, const int32_t* coords, int64_t N, const Codec& cin,
                  Transient& tr, int32_t* copy_out) {
  const uint64_t slots = tr.table.nbuckets * 4;
  k_fill_u64<<<grid_for(static_cast<int64_t>(slots / 4), kBlock), kBlock, 0, rb->stream>>>(
      tr.table.slots, kEmpty, slots);
  if (N == 0) return SPCONV_OK;
  if (tr.wide)
    k_insert<true><<<grid_for(N), kBlock, 0, rb->stream>>>(coords, N, cin, tr.table, tr.keys,
                                                           copy_out, &rb->hdr->status);
  else
    k_insert<false><<<grid_for(N), kBlock, 0, rb->stream>>>(coords, N, cin, tr.table, tr.keys,
                                                            copy_out, &rb->hdr->status);
  return SPCONV_OK;
}

// Per-offset pair counts -> k_i and pair_off; gather map -> pair lists.
// (Small books, at most kSelfScan words of counts read over all blocks: the
// compaction sums the counts itself, one launch instead of two.)
constexpr int64_t kSelfScan = int64_t{1} << 22;
void launch_scan_compact(spconv_rulebook rb) {
  const bool self = rb->K * rb->nblk * rb->nblk <= kSelfScan;
  if (!self)
    k_scan<<<static_cast<unsigned>(rb->K), kBlock, 0, rb->stream>>>(rb->blk_cnt, rb->nblk,
                                                                    rb->totals);
  (self ? k_compact<true> : k_compact<false>)<<<static_cast<unsigned>(rb->nblk), kBlock, 0,
                                               rb->stream>>>(
      rb->gmap, rb->perm, rb->blk_cnt, rb->wpre, rb->totals, static_cast<int>(rb->K), rb->gstride,
      rb->n_cap, rb->hdr, rb->nblk, reinterpret_cast<int2*>(rb->pairs), rb->pair_off);
}

void launch_probe_scan_compact(spconv_rulebook rb, const uint64_t* rowkeys, const Codec& crow,
                               const Codec& cin, const Transient& tr) {
  const OffsetTable ot = make_offsets(rb);
  const unsigned g = probe_grid_size(rb->nblk);
  auto launch = [&](auto kern) {
    kern<<<g, kBlock, 0, rb->stream>>>(rowkeys, rb->perm, rb->hdr, rb->gstride, crow, cin,
                                       tr.table, ot, rb->gmap, rb->blk_cnt, rb->wpre, rb->nblk);
  };
  const bool sc = rb->kind == SPCONV_SC;
#define SPC_PROBE(W, S)                                      \
  switch (rb->D) {                                           \
    case 2: launch(k_probe<W, S, 2>); break;                 \
    case 3: launch(k_probe<W, S, 3>); break;                 \
    default: launch(k_probe<W, S, 4>); break;                \
  }
  if (tr.wide) {
    if (sc) { SPC_PROBE(true, true) } else { SPC_PROBE(true, false) }
  } else {
    if (sc) { SPC_PROBE(false, true) } else { SPC_PROBE(false, false) }
  }
#undef SPC_PROBE
  launch_scan_compact(rb);
}

// Geometry of the brick map for a VSC book, or false where it does not apply:
// bricks of up to 64 cells (b = 6 / d bits per coordinate, fewer where a
// coordinate has fewer), every coordinate's brick side at least f_j - 1 (so
// a neighbour crosses at most one face per coordinate), at most kBrickK
// offsets.  SPCONV_RULEBOOK=table, SPCONV_HASH_LAYOUT and
// SPCONV_TEST_HASH_SLOTS keep the open-addressing table of sites instead.
bool brick_geom(spconv_rulebook rb, BrickMap* m) {
  if (rb->kind != SPCONV_VSC || rb->K > kBrickK || rb->in_count) return false;
  if (std::getenv("SPCONV_HASH_LAYOUT") || std::getenv("SPCONV_TEST_HASH_SLOTS")) return false;
  if (const char* e = std::getenv("SPCONV_RULEBOOK"))
    if (std::strcmp(e, "table") == 0) return false;
  *m = BrickMap{};
  m->D = rb->D;
  const int d = rb->D - 1;
  const int b = 6 / d;
  int bits[kMaxD] = {0, 0, 0, 0}, maxb = 0, B = 0;
  for (int j = 1; j < rb->D; ++j) {
    bits[j] = bitlen(static_cast<uint64_t>(rb->size[j] - 1));
    maxb = bits[j] > maxb ? bits[j] : maxb;
    B += bits[j];
  }
  if (B + bitlen(static_cast<uint64_t>(rb->size[0] - 1)) > 63) return false;
  // cell bits: lowest = level 0 of the last coordinate, coordinate 1 on top
  // inside a level (the order of the schedule's Morton codes)
  int pos = 0;
  for (int L = 0; L < maxb; ++L)
    for (int j = rb->D - 1; j >= 1; --j)
      if (bits[j] > L) m->M[j] |= 1ull << pos++;
  m->lb = 0;
  for (int j = 1; j < rb->D; ++j) {
    const int bj = bits[j] < b ? bits[j] : b;
    m->side[j] = 1 << bj;
    m->lb += bj;
    if (m->side[j] < rb->f[j] - 1) return false;
  }
  if (m->lb < 2) return false;     // a brick is written in 16-byte pieces
  const uint64_t lowmask = (1ull << m->lb) - 1;
  for (int j = 1; j < rb->D; ++j) m->BM[j] = (m->M[j] & ~lowmask) >> m->lb;
  return true;
}

// VSC book on the brick map: keys, the Morton schedule (sorted), brick runs,
// directory and pool, then the probe, scan and compaction.
int build_vsc_bricks(spconv_rulebook rb, const int32_t* coords, BrickMap m) {
  const int64_t N = rb->n_in;
  const Codec cin = make_codec(rb->D, rb->size);
  k_init_header<<<1, 64, 0, rb->stream>>>(rb->hdr, N);
  uint64_t dslots = 64;
  while (dslots < 2 * static_cast<uint64_t>(N)) dslots <<= 1;
  const int64_t nb = rb->nblk;
  const size_t bytes = align_up(N * 8, 256) + schedule_bytes(rb->n_cap) +
                       2 * align_up(static_cast<size_t>(nb) * kBlock / 8, 256) +
                       align_up(static_cast<size_t>(nb) * 4, 256) + 256 +
                       align_up(dslots * 16, 256) +
                       align_up((static_cast<size_t>(N) << m.lb) * 4, 256) +
                       align_up(static_cast<size_t>(N) * 4, 256) +
                       align_up(static_cast<size_t>(N) * 8, 256) +
                       align_up(static_cast<size_t>(N) * 27 * 4, 256) +
                       align_up(static_cast<size_t>(kBrickCells) * kBrickK * 2, 256) + 256;
  void* mem = nullptr;
  if (dev_alloc(rb, bytes, rb->stream, &mem) != SPCONV_OK) return SPCONV_ENOMEM;
  Carver cv{static_cast<char*>(mem)};
  uint64_t* keys = cv.take<uint64_t>(N);
  uint64_t* flagbits = cv.take<uint64_t>(static_cast<size_t>(nb) * (kBlock / kWave));
  uint64_t* validbits = cv.take<uint64_t>(static_cast<size_t>(nb) * (kBlock / kWave));
  uint32_t* bsum = cv.take<uint32_t>(static_cast<size_t>(nb));
  DeviceHeader* bh = cv.take<DeviceHeader>(1);
  m.dir = cv.take<ulonglong2>(dslots);
  m.dslots = dslots;
  m.pool = cv.take<int32_t>(static_cast<size_t>(N) << m.lb);
  m.nbricks = bh;
  int32_t* brickidx = cv.take<int32_t>(N);
  int64_t* starts = cv.take<int64_t>(N);
  int nb3 = 1;
  for (int j = 1; j < rb->D; ++j) nb3 *= 3;
  int32_t* nbr = cv.take<int32_t>(static_cast<size_t>(N) * nb3);
  uint16_t* tab = cv.take<uint16_t>(static_cast<size_t>(kBrickCells) * kBrickK);
  // keys and Morton codes in one pass; sorted by brick only (k_pool_fill
  // puts each brick's sites in cell order)
  const SiteIn si{coords, N, keys, rb->out_coords, &rb->hdr->status};
  uint64_t* mk = const_cast<uint64_t*>(launch_schedule(rb, keys, cin, &cv, m.lb, &si));
  const OffsetTable ot = make_offsets(rb);
  const int64_t ntab = (int64_t{1} << m.lb) * ot.K;
  const int64_t fb = nb > (ntab + kBlock - 1) / kBlock ? nb : (ntab + kBlock - 1) / kBlock;
  k_brick_flags<<<static_cast<unsigned>(fb), kBlock, 0, rb->stream>>>(
      mk, rb->perm, keys, N, nb, m.lb, flagbits, validbits, bsum, &rb->hdr->status, ot, m, tab);
  k_bitscan<<<1, kBlock, 0, rb->stream>>>(bsum, nb, bh, -1, nullptr);
  const unsigned gb = static_cast<unsigned>(nb < kPoolBlocks ? nb : kPoolBlocks);
  k_dir_clear<<<gb, kBlock, 0, rb->stream>>>(m, nbr, nb3);
  k_bricks<<<static_cast<unsigned>(nb), kBlock, 0, rb->stream>>>(mk, rb->perm, N, flagbits,
                                                                 validbits, bsum, m, brickidx,
                                                                 starts);
  k_pool_fill<<<gb, kBlock, 0, rb->stream>>>(mk, rb->perm, validbits, N, starts, m,
                                              &rb->hdr->status);
  k_brick_nbrs<<<gb, kBlock, 0, rb->stream>>>(mk, starts, cin, m, nb3, nbr);
  const unsigned g = probe_grid_size(rb->nblk);
  auto launch = [&](auto kern) {
    kern<<<g, kBlock, 0, rb->stream>>>(mk, rb->perm, brickidx, keys, rb->hdr, rb->gstride, cin,
                                       ot, m, tab, nbr, nb3, rb->gmap, rb->blk_cnt, rb->wpre,
                                       rb->nblk);
  };
  switch (rb->D) {
    case 2: launch(k_probe_brick<2>); break;
    case 3: launch(k_probe_brick<3>); break;
    default: launch(k_probe_brick<4>); break;
  }
  launch_scan_compact(rb);
  if (dev_free(rb, mem, rb->stream) != SPCONV_OK) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

int finish(spconv_rulebook rb, Transient& tr) {
  if (dev_free(rb, tr.mem, rb->stream) != SPCONV_OK) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}


// Dense-grid geometry of a grid with extents `size` (coordinate 0 = sample).
// False unless it has fewer than kGridMaxCells cells (grid bytes must stay
// below 2^31 for the probe's buffer loads).
constexpr uint64_t kGridMaxCells = 1ull << 29;

bool make_grid_geom(int D, const int32_t* size, GridGeom* g, uint64_t* cells) {
  *g = GridGeom{};
  g->D = D;
  int bits[kMaxD] = {0, 0, 0, 0};
  int maxb = 0;
  for (int j = 0; j < D; ++j) g->size[j] = size[j];
  for (int j = 1; j < D; ++j) {
    bits[j] = bitlen(static_cast<uint64_t>(size[j] - 1));
    maxb = bits[j] > maxb ? bits[j] : maxb;
    g->B += bits[j];
  }
  // lowest Z bit = level 0 of the last coordinate; coordinate 1 is the most
  // significant inside every level
  int pos = 0;
  for (int L = 0; L < maxb; ++L)
    for (int j = D - 1; j >= 1; --j)
      if (bits[j] > L) g->M[j] |= 1u << pos++;
  if (g->B > 29) return false;
  *cells = static_cast<uint64_t>(size[0]) << g->B;
  return *cells < kGridMaxCells;
}

// Dense grid or hash table for the input sites.  The grid costs memory
// traffic per cell of its power-of-two padded extent (clearing it, deriving
// its bitmap), the hash table latency-bound work per site plus a fixed
// ~170 us of sorting and compaction.  Measured on surfaces (VSC 3^3 and SC
// 2^3/2 builds), the two cross between 400 and 600 padded cells per site, so
// the grid is taken while it has at most 400 cells per site (plus 4M cells
// for small inputs).  SPCONV_RULEBOOK=hash / =grid forces a choice.
bool use_grid(uint64_t cells, int64_t N) {
  if (const char* e = std::getenv("SPCONV_RULEBOOK")) {
    if (std::strcmp(e, "hash") == 0 || std::strcmp(e, "table") == 0) return false;
    if (std::strcmp(e, "grid") == 0) return true;
  }
  return cells <= 400ull * static_cast<uint64_t>(N) + (1ull << 22);
}

struct GridBufs {
  uint32_t* grid;     // [cells] 1 + row, 0 = empty
  uint32_t* bitmap;   // [nwords] occupancy (right after the grid)
  uint32_t* bsum;     // [nbw] occupied cells per 256 words, then their bases
  bool self;          // small: the scatter sets the bitmap, one launch schedules
  uint64_t nwords;
  int64_t nbw;
};

// Whether a grid of `cells` cells is scheduled by one launch
// (k_grid_emit_self, the bitmap set by the scatter) rather than by three.
bool self_schedule(uint64_t cells) {
  if (const char* e = std::getenv("SPCONV_RULEBOOK"))
    if (std::strcmp(e, "grid3") == 0) return false;    // test knob: the three-launch schedule
  return (cells + 31) / 32 <= static_cast<uint64_t>(kSelfWords);
}

size_t grid_bytes(uint64_t cells) {
  const uint64_t nwords = (cells + 31) / 32;
  const uint64_t nbw = (nwords + kBlock - 1) / kBlock;
  return align_up(cells * 4, 256) + align_up(nwords * 4, 256) + align_up(nbw * 4, 256);
}

// sched: the grid will give a schedule.
GridBufs take_grid(Carver* cv, uint64_t cells, bool sched = false) {
  GridBufs b{};
  b.nwords = (cells + 31) / 32;
  b.nbw = static_cast<int64_t>((b.nwords + kBlock - 1) / kBlock);
  b.grid = cv->take<uint32_t>(cells);
  b.bitmap = cv->take<uint32_t>(b.nwords);
  b.bsum = cv->take<uint32_t>(static_cast<size_t>(b.nbw));
  b.self = sched && self_schedule(cells);
  return b;
}

// Clear the grid and scatter rows [0, N) (or [0, *count)) into it; `cas`
// detects duplicates at the scatter, otherwise the schedule's count does.
// init_n >= 0 also initialises the header with n_out = init_n.
void launch_grid_scatter(spconv_rulebook rb, const int32_t* coords, int64_t N,
                         const int64_t* count, const GridGeom& g, uint64_t cells,
                         const GridBufs& b, int32_t* copy_out, const Codec& ckey,
                         uint64_t* keys_out, bool cas, int64_t init_n = -1) {
  // with a one-launch schedule the scatter sets the bitmap as well, which
  // lies right after the grid and is cleared with it
  const uint64_t nclear = b.self ? static_cast<uint64_t>(b.bitmap + b.nwords - b.grid) : cells;
  launch_zero(b.grid, nclear, rb->stream, init_n >= 0 ? rb->hdr : nullptr, init_n);
  auto kern = cas ? k_grid_scatter<true> : k_grid_scatter<false>;
  // a book on another book's outputs keeps its own copy of their count
  int64_t* cc = count && count == rb->in_count ? rb->n_in_dev : nullptr;
  kern<<<grid_for(N), kBlock, 0, rb->stream>>>(coords, N, count, g, b.grid, copy_out, ckey,
                                               keys_out, &rb->hdr->status, cc,
                                               b.self ? b.bitmap : nullptr);
}

// Z-order schedule from the grid; also sets n_out to the number of occupied
// cells, flagging duplicates when that is not `expect` (>= 0).
void launch_grid_schedule(spconv_rulebook rb, const GridBufs& b, uint64_t cells,
                          int64_t expect, const int64_t* expect_dev = nullptr) {
  if (b.self) {
    k_grid_emit_self<<<static_cast<unsigned>(b.nbw * kEmitParts), kBlock, 0, rb->stream>>>(
        b.bitmap, b.nwords, cells, b.grid, rb->perm, rb->hdr, expect, expect_dev);
    return;
  }
  k_grid_bits<<<static_cast<unsigned>(b.nbw), kBlock, 0, rb->stream>>>(b.grid, cells, b.nwords,
                                                                        b.bitmap, b.bsum);
  if (b.nbw <= kSelfBlocks) {
    k_grid_emit<true><<<static_cast<unsigned>(b.nbw), kBlock, 0, rb->stream>>>(
        b.bitmap, b.nwords, cells, b.bsum, b.grid, rb->perm, rb->hdr, expect, expect_dev);
    return;
  }
  k_bitscan<<<1, kBlock, 0, rb->stream>>>(b.bsum, b.nbw, rb->hdr, expect, expect_dev);
  k_grid_emit<false><<<static_cast<unsigned>(b.nbw), kBlock, 0, rb->stream>>>(
      b.bitmap, b.nwords, cells, b.bsum, b.grid, rb->perm, rb->hdr, expect, expect_dev);
}

void launch_probe_grid(spconv_rulebook rb, const int32_t* rows_sites, const GridGeom& g,
                       const GridBufs& b, uint64_t cells) {
  const OffsetTable ot = make_offsets(rb);
  auto launch = [&](auto kern) {
    kern<<<probe_grid_size(rb->nblk), kBlock, 0, rb->stream>>>(
        rows_sites, rb->perm, rb->hdr, rb->gstride, g, ot, b.grid, static_cast<uint32_t>(cells),
        rb->gmap, rb->blk_cnt, rb->wpre, rb->nblk);
  };
  const bool sc = rb->kind == SPCONV_SC;
  if (!sc && rb->D == 4 && rb->f[1] == 3 && rb->f[2] == 3 && rb->f[3] == 3 &&
      (g.M[3] & 1u) && (g.M[2] & 2u)) {
    // count, scan the counts into block bases, then write the gather map and
    // the pairs in one pass (no compaction kernel re-reading the gather map)
    auto probe = [&](auto kern) {
      kern<<<probe_grid_size(rb->nblk), kBlock, 0, rb->stream>>>(
          rows_sites, rb->perm, rb->hdr, rb->gstride, g, b.grid, static_cast<uint32_t>(cells),
          b.bitmap, rb->gmap, rb->blk_cnt, rb->wpre, rb->nblk, rb->totals,
          reinterpret_cast<int2*>(rb->pairs), rb->pair_off);
    };
    probe(k_probe_grid_g4<false>);
    k_scan<<<static_cast<unsigned>(rb->K), kBlock, 0, rb->stream>>>(rb->blk_cnt, rb->nblk,
                                                                    rb->totals);
    probe(k_probe_grid_g4<true>);
    return;
  }
  if (sc && rb->D == 4 && rb->f[1] == 2 && rb->f[2] == 2 && rb->f[3] == 2 && rb->s[1] == 2 &&
      rb->s[2] == 2 && rb->s[3] == 2 && (g.M[3] & 1u) && (g.M[2] & 2u) && (g.M[1] & 4u)) {
    k_probe_grid_sc2<<<probe_grid_size(rb->nblk), kBlock, 0, rb->stream>>>(
        rows_sites, rb->perm, rb->hdr, rb->gstride, g, b.grid, static_cast<uint32_t>(cells),
        rb->gmap, rb->blk_cnt, rb->wpre, rb->nblk);
    launch_scan_compact(rb);
    return;
  }
#define SPC_PROBE(S)                                         \
  switch (rb->D) {                                           \
    case 2: launch(k_probe_grid<S, 2>); break;               \
    case 3: launch(k_probe_grid<S, 3>); break;               \
    default: launch(k_probe_grid<S, 4>); break;              \
  }
  if (sc) { SPC_PROBE(true) } else { SPC_PROBE(false) }
#undef SPC_PROBE
  launch_scan_compact(rb);
}

int build_vsc_grid(spconv_rulebook rb, const int32_t* coords, const GridGeom& g,
                   uint64_t cells) {
  const int64_t N = rb->n_in;
  void* mem = nullptr;
  if (dev_alloc(rb, grid_bytes(cells) + 256, rb->stream, &mem) != SPCONV_OK)
    return SPCONV_ENOMEM;
  Carver cv{static_cast<char*>(mem)};
  const GridBufs b = take_grid(&cv, cells, true);
  // rows [0, N), or [0, *in_count) for a book on another book's outputs
  launch_grid_scatter(rb, coords, N, rb->in_count, g, cells, b, rb->out_coords, Codec{}, nullptr,
                      false, rb->in_count ? 0 : N);
  launch_grid_schedule(rb, b, cells, rb->in_count ? -1 : N, rb->in_count);
  launch_probe_grid(rb, rb->out_coords, g, b, cells);
  if (dev_free(rb, mem, rb->stream) != SPCONV_OK) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

// SC on dense grids: input sites scattered into the input grid and, in the
// same pass, the output set marked in a lexicographic bitmap over the output
// grid; the bitmap ranked (rows in lexicographic order), and the emission of
// the output sites fills the output grid, whose occupancy gives the Z-order
// schedule.  Everything that must start at zero (input grid, lexicographic
// bitmap, output grid and, for a one-launch schedule, its bitmap) is laid
// out in one range and cleared by one launch.
int build_sc_grid(spconv_rulebook rb, const int32_t* coords, const GridGeom& gi,
                  uint64_t cells_in, const GridGeom& go, uint64_t cells_out) {
  const int64_t N = rb->n_in;
  const Codec cout = make_codec(rb->D, rb->out_size);
  uint64_t lex_cells = 1;
  for (int j = 0; j < rb->D; ++j) lex_cells *= static_cast<uint64_t>(rb->out_size[j]);
  const uint64_t lwords = (lex_cells + 31) / 32;
  const int64_t lnbw = static_cast<int64_t>((lwords + kBlock - 1) / kBlock);
  const size_t bytes = align_up(cells_in * 4, 256) +
                       align_up(lwords * 4, 256) + grid_bytes(cells_out) +
                       align_up(static_cast<size_t>(lnbw) * 4, 256) + 256;
  void* mem = nullptr;
  if (dev_alloc(rb, bytes, rb->stream, &mem) != SPCONV_OK) return SPCONV_ENOMEM;
  Carver cv{static_cast<char*>(mem)};
  GridBufs bi{};
  bi.grid = cv.take<uint32_t>(cells_in);
  uint32_t* lex = cv.take<uint32_t>(lwords);
  const GridBufs bo = take_grid(&cv, cells_out, true);
  uint32_t* lsum = cv.take<uint32_t>(static_cast<size_t>(lnbw));
  uint32_t* from = bi.grid;
  uint32_t* to = bo.self ? bo.bitmap + bo.nwords : bo.grid + cells_out;
  launch_zero(from, static_cast<uint64_t>(to - from), rb->stream, rb->hdr, 0);
  Extents E{};
  for (int j = 0; j < rb->D; ++j) E.e[j] = rb->out_size[j];
  const OffsetTable ot = make_offsets(rb);
  // a book on another book's outputs keeps its own copy of their count
  int64_t* cc = rb->in_count ? rb->n_in_dev : nullptr;
  k_sc_scatter_mark<<<grid_for(N), kBlock, 0, rb->stream>>>(
      coords, N, rb->in_count, gi, bi.grid, &rb->hdr->status, cc, ot, E, lex);
  const bool lself = lwords <= static_cast<uint64_t>(kSelfWords);
  if (!lself) {
    k_bitsum<<<static_cast<unsigned>(lnbw), kBlock, 0, rb->stream>>>(lex, lwords, lsum);
    k_bitscan<<<1, kBlock, 0, rb->stream>>>(lsum, lnbw, rb->hdr, -1, nullptr);
  }
  const OutGrid og{go, bo.grid, bo.self ? bo.bitmap : nullptr};
  k_sc_emit<<<static_cast<unsigned>(lnbw * kEmitParts), kBlock, 0, rb->stream>>>(
      lex, lwords, lself ? nullptr : lsum, cout, E, rb->out_coords, nullptr, og, rb->hdr);
  launch_grid_schedule(rb, bo, cells_out, -1, nullptr);
  launch_probe_grid(rb, rb->out_coords, gi, bi, cells_in);
  if (dev_free(rb, mem, rb->stream) != SPCONV_OK) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}
}  // namespace

__global__ void k_copy_count(int64_t* __restrict__ dst, const int64_t* __restrict__ src) {
  if (threadIdx.x == 0) *dst = *src;
}

void copy_in_count(spconv_rulebook rb) {
  k_copy_count<<<1, 64, 0, rb->stream>>>(rb->n_in_dev, rb->in_count);
}

bool grid_build(spconv_rulebook rb) {
  const int64_t N = rb->n_in;
  GridGeom g, go;
  uint64_t ci = 0, co = 0;
  if (N <= 0 || !make_grid_geom(rb->D, rb->size, &g, &ci) || !use_grid(ci, N)) return false;
  if (rb->kind == SPCONV_VSC) return true;
  for (int j = 0; j < rb->D; ++j)
    if (rb->out_size[j] <= 0) return false;
  return make_grid_geom(rb->D, rb->out_size, &go, &co);
}

// Whether a VSC build takes the one-workgroup path: a few sites on a few
// cells (*sbits = spatial bits of a cell number, *nwords = bitmap words), a
// site count known on the host (not a book chained on device counts), and no
// site map forced by SPCONV_RULEBOOK (=small forces it where it applies).
bool small_build(spconv_rulebook rb, int* sbits, int* nwords) {
  const int64_t N = rb->n_in;
  if (rb->in_count || N <= 0 || N > kSmallN || rb->K > kSmallK) return false;
  int B = 0;                       // 2^B >= extent + (f - 1) / 2 in every dimension
  for (int j = 1; j < rb->D; ++j) {
    const int64_t span = int64_t{rb->size[j]} + (rb->f[j] - 1) / 2;
    while ((int64_t{1} << B) < span) ++B;
  }
  if (B > kSmallCellBits) return false;
  *sbits = (rb->D - 1) * B;
  if (*sbits > kSmallCellBits) return false;
  const uint64_t cells = static_cast<uint64_t>(rb->size[0]) << *sbits;
  if (cells > (uint64_t{1} << kSmallCellBits)) return false;
  *nwords = static_cast<int>((cells + 31) / 32);
  if (const char* e = std::getenv("SPCONV_RULEBOOK")) return std::strcmp(e, "small") == 0;
  return true;
}

int build_vsc(spconv_rulebook rb, const int32_t* coords) {
  const int64_t N = rb->n_in;
  int sbits = 0, nwords = 0;
  if (small_build(rb, &sbits, &nwords)) {
    Extents E{};
    for (int j = 0; j < rb->D; ++j) E.e[j] = rb->size[j];
    auto launch = [&](auto kern) {
      kern<<<1, kSmallThreads, 0, rb->stream>>>(
          coords, static_cast<int>(N), sbits, nwords, make_offsets(rb), E, rb->out_coords, rb->perm, rb->gmap,
          rb->gstride, rb->blk_cnt, rb->nblk, rb->totals, rb->pair_off,
          reinterpret_cast<int2*>(rb->pairs), rb->hdr);
    };
    switch (rb->D) {
      case 2: launch(k_build_small<2>); break;
      case 3: launch(k_build_small<3>); break;
      default: launch(k_build_small<4>); break;
    }
    return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
  }
  GridGeom g;
  uint64_t cells = 0;
  if (N > 0 && make_grid_geom(rb->D, rb->size, &g, &cells) && use_grid(cells, N))
    return build_vsc_grid(rb, coords, g, cells);
  BrickMap bm;
  if (N > 0 && brick_geom(rb, &bm)) return build_vsc_bricks(rb, coords, bm);
  const Codec cin = make_codec(rb->D, rb->size);
  k_init_header<<<1, 64, 0, rb->stream>>>(rb->hdr, N);
  Transient tr;
  Carver cv;
  int st = alloc_transient(rb, N, cin, schedule_bytes(rb->n_cap), &tr, &cv);
  if (st != SPCONV_OK) return st;
  launch_insert(rb, coords, N, cin, tr, rb->out_coords);
  if (N > 0) {
    launch_schedule(rb, tr.keys, cin, &cv, 0, nullptr);
    launch_probe_scan_compact(rb, tr.keys, cin, cin, tr);
  }
  else
    k_fill_u64<<<1, 64, 0, rb->stream>>>(reinterpret_cast<uint64_t*>(rb->pair_off), 0,
                                         static_cast<uint64_t>(rb->K + 1));
  return finish(rb, tr);
}

int build_sc(spconv_rulebook rb, const int32_t* coords) {
  const int64_t N = rb->n_in;
  {
    GridGeom gi, go;
    uint64_t ci = 0, co = 0;
    bool any_out = true;
    for (int j = 0; j < rb->D; ++j) any_out = any_out && rb->out_size[j] > 0;
    if (N > 0 && any_out && make_grid_geom(rb->D, rb->size, &gi, &ci) &&
        make_grid_geom(rb->D, rb->out_size, &go, &co) && use_grid(ci, N))
      return build_sc_grid(rb, coords, gi, ci, go, co);
  }
  const Codec cin = make_codec(rb->D, rb->size);
  const Codec cout = make_codec(rb->D, rb->out_size);
  uint64_t cells = 1;
  for (int j = 0; j < rb->D; ++j) cells *= static_cast<uint64_t>(rb->out_size[j]);
  const uint64_t nwords = (cells + 31) / 32;
  const int64_t nbw = static_cast<int64_t>((nwords + kBlock - 1) / kBlock);
  k_init_header<<<1, 64, 0, rb->stream>>>(rb->hdr, 0);
  const size_t extra = align_up(nwords * 4, 256) + align_up(nbw * 4, 256) +
                       align_up(static_cast<size_t>(rb->n_cap) * 8, 256) +
                       schedule_bytes(rb->n_cap);
  Transient tr;
  Carver cv;
  int st = alloc_transient(rb, N, cin, extra, &tr, &cv);
  if (st != SPCONV_OK) return st;
  uint32_t* bitmap = cv.take<uint32_t>(nwords);
  uint32_t* bsum = cv.take<uint32_t>(nbw);
  uint64_t* out_keys = cv.take<uint64_t>(rb->n_cap);
  Extents E{};
  for (int j = 0; j < rb->D; ++j) E.e[j] = rb->out_size[j];
  launch_insert(rb, coords, N, cin, tr, nullptr);
  if (N > 0 && cells > 0) {
    k_fill_u32<<<grid_for(static_cast<int64_t>(nwords)), kBlock, 0, rb->stream>>>(bitmap, 0u,
                                                                               nwords);
    const OffsetTable ot = make_offsets(rb);
    k_sc_mark<<<grid_for(N), kBlock, 0, rb->stream>>>(tr.keys, N, nullptr, cin, ot, E, bitmap);
    k_bitsum<<<static_cast<unsigned>(nbw), kBlock, 0, rb->stream>>>(bitmap, nwords, bsum);
    k_bitscan<<<1, kBlock, 0, rb->stream>>>(bsum, nbw, rb->hdr, -1, nullptr);
    k_sc_emit<<<static_cast<unsigned>(nbw * kEmitParts), kBlock, 0, rb->stream>>>(
        bitmap, nwords, bsum, cout, E, rb->out_coords, out_keys, OutGrid{}, rb->hdr);
    launch_schedule(rb, out_keys, cout, &cv, 0, nullptr);
    launch_probe_scan_compact(rb, out_keys, cout, cin, tr);
  } else {
    k_fill_u64<<<1, 64, 0, rb->stream>>>(reinterpret_cast<uint64_t*>(rb->pair_off), 0,
                                         static_cast<uint64_t>(rb->K + 1));
  }
  return finish(rb, tr);
}

}  // namespace spc
