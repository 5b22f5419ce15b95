// Sparse pooling, the transposed rule book, and the weight / bias gradients
// on gfx950.
//
// Pooling (Section 3 defines max-pooling MP(f,s) and average-pooling AP(f,s)
// as variants of SC(.,.,f,s)): one lane per (output position, 16-byte chunk
// of channels) walks the offsets of the SC gather map in ascending order;
// MP starts from the zero vector and takes IEEE maxNum (exact in any dtype),
// AP sums in fp32 and divides by prod_j f_j once.
//
// Transposed rule book (Section 3: DC(.,.,f,s) inverts SC(.,.,f,s), same
// connections reversed; the SC input gradient runs the same reversed pairs):
//   k_class_keys + radix sort  SC input rows ordered by their offset class
//                              x mod s (stable, so by row inside a class):
//                              with f = s every row of a class takes the same
//                              single offset, so 16-row blocks stay uniform
//   k_inverse                  position of every row in that order
//   k_fill_i32 + k_scatter_transpose
//                              G^T[i][q] = 1 + SC output row of the pair of R_i
//                              whose input row sits at position q (each
//                              (offset, input row) has at most one pair)
// The output-stationary forward kernels then run DC and the input gradients
// over this map.  When f = s every SC input row has exactly one pair, and
// the rule book also keeps R_i split into its two columns (source rows + 1,
// destination rows), each offset's run padded to whole chunks of kSegRows:
//   k_chunk_layout, k_seg_fill, k_seg_scatter
// so DC and the SC input gradient run as one gather-multiply-store launch
// (the forward kernels with one offset, W^i chosen per chunk), with no empty
// offsets to walk.
//
// Weight gradient dW^i = sum over the pairs of R_i of (input row)^T x (output
// gradient row): the output positions of the rule book's schedule are cut
// into chunks of kChunk positions, and chunk c of R_i is its pairs whose
// output lies in chunk c (at most kChunk of them); one workgroup forms
// the fp32 partial product of a chunk for a 64x64 tile of dW^i (bf16: on the
// matrix cores, pairs gathered row-major into LDS and read back transposed;
// fp32 and odd widths: vector ALU, 4x4 outputs per lane), and a second kernel
// adds the chunks of every entry in ascending chunk order.  The bias
// gradient sums the output-gradient rows in fixed row chunks the same way.
// No atomics anywhere: results are bitwise reproducible.
#include "internal.h"

namespace spc {
namespace {

__device__ __forceinline__ float bf16f(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T> struct IO;
template <> struct IO<float> {
  static constexpr int kVec = 4;
  __device__ static float ld(const float* p, int64_t i) { return p[i]; }
  __device__ static void st(float* p, int64_t i, float v) { p[i] = v; }
  __device__ static void ld16(const float* p, int64_t i, float* v) {
    const float4 q = *reinterpret_cast<const float4*>(p + i);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  }
  __device__ static void st16(float* p, int64_t i, const float* v) {
    *reinterpret_cast<float4*>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct IO<uint16_t> {
  static constexpr int kVec = 8;
  __device__ static float ld(const uint16_t* p, int64_t i) { return bf16f(p[i]); }
  __device__ static void st(uint16_t* p, int64_t i, float v) { p[i] = to_bf16(v); }
  __device__ static void ld16(const uint16_t* p, int64_t i, float* v) {
    const uint4 q = *reinterpret_cast<const uint4*>(p + i);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(w[e] << 16);
      v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  }
  __device__ static void st16(uint16_t* p, int64_t i, const float* v) {
    uint4 q;
    q.x = to_bf16(v[0]) | (static_cast<uint32_t>(to_bf16(v[1])) << 16);
    q.y = to_bf16(v[2]) | (static_cast<uint32_t>(to_bf16(v[3])) << 16);
    q.z = to_bf16(v[4]) | (static_cast<uint32_t>(to_bf16(v[5])) << 16);
    q.w = to_bf16(v[6]) | (static_cast<uint32_t>(to_bf16(v[7])) << 16);
    *reinterpret_cast<uint4*>(p + i) = q;
  }
};

inline unsigned grid_of(int64_t n, int64_t cap = 65536) {
  int64_t b = (n + 255) / 256;
  if (b > cap) b = cap;
  return static_cast<unsigned>(b < 1 ? 1 : b);
}

// ---------------------------------------------------------------------------
// Pooling
// ---------------------------------------------------------------------------
// Thread = (output position, VEC channels).  The gather-map entries of 8
// offsets are loaded together, then their input rows (an absent neighbour
// reads row 0 and is not taken), so the loads of a batch are in flight at
// once instead of one offset after another behind a branch; the rows are
// taken in ascending offset order.
template <typename T, int VEC, bool MAX>
__global__ __launch_bounds__(256) void k_pool(const int32_t* __restrict__ gmap,
                                              const int32_t* __restrict__ perm, int64_t gstride,
                                              const DeviceHeader* __restrict__ hdr, int K,
                                              const T* __restrict__ x, T* __restrict__ y, int C) {
  constexpr int KB = 8;
  const int nch = C / VEC;
  const int64_t total = hdr->n_out * nch;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t idx = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; idx < total;
       idx += stride) {
    const int64_t p = idx / nch;
    const int c0 = static_cast<int>(idx - p * nch) * VEC;
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.0f;   // MP: the zero vector; AP: empty sum
    for (int i0 = 0; i0 < K; i0 += KB) {
      int32_t g[KB];
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const int i = i0 + u < K ? i0 + u : K - 1;
        g[u] = gmap[i * gstride + p] - 1;
      }
#pragma unroll
      for (int u = 0; u < KB; ++u) g[u] = i0 + u < K ? g[u] : -1;
      float v[KB][VEC];
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        const int64_t base = static_cast<int64_t>(g[u] >= 0 ? g[u] : 0) * C + c0;
        if constexpr (VEC == 1) {
          v[u][0] = IO<T>::ld(x, base);
        } else {
          IO<T>::ld16(x, base, v[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < KB; ++u) {
        if (g[u] < 0) continue;
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = MAX ? fmaxf(acc[e], v[u][e]) : acc[e] + v[u][e];
      }
    }
    if constexpr (!MAX) {
      const float k = static_cast<float>(K);
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = acc[e] / k;
    }
    const int64_t ob = static_cast<int64_t>(perm[p]) * C + c0;
    if constexpr (VEC == 1) {
      IO<T>::st(y, ob, acc[0]);
    } else {
      IO<T>::st16(y, ob, acc);
    }
  }
}

template <typename T, bool MAX>
void launch_pool(spconv_rulebook rb, const void* x, void* y, int C, hipStream_t st) {
  const bool vec = C % IO<T>::kVec == 0;
  const int64_t work = rb->n_cap * (vec ? C / IO<T>::kVec : C);
  if (vec)
    k_pool<T, IO<T>::kVec, MAX><<<grid_of(work), 256, 0, st>>>(
        rb->gmap, rb->perm, rb->gstride, rb->hdr, static_cast<int>(rb->K),
        static_cast<const T*>(x), static_cast<T*>(y), C);
  else
    k_pool<T, 1, MAX><<<grid_of(work), 256, 0, st>>>(
        rb->gmap, rb->perm, rb->gstride, rb->hdr, static_cast<int>(rb->K),
        static_cast<const T*>(x), static_cast<T*>(y), C);
}

// ---------------------------------------------------------------------------
// Transposed rule book
// ---------------------------------------------------------------------------
struct ClassGeom {
  int D;
  int32_t s[kMaxD];
  int64_t mult[kMaxD];   // class = sum_j (x_j mod s_j) mult_j, last dimension fastest
};

__global__ __launch_bounds__(256) void k_class_keys(const int32_t* __restrict__ coords, int64_t n,
                                                    ClassGeom g, uint64_t* __restrict__ keys,
                                                    int32_t* __restrict__ vals) {
  const int64_t r = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (r >= n) return;
  uint64_t c = 0;
  for (int j = 1; j < g.D; ++j)
    c += static_cast<uint64_t>(coords[r * g.D + j] % g.s[j]) * static_cast<uint64_t>(g.mult[j]);
  keys[r] = c;
  vals[r] = static_cast<int32_t>(r);
}

__global__ __launch_bounds__(256) void k_iota(int32_t* __restrict__ a, int64_t n) {
  const int64_t r = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (r < n) a[r] = static_cast<int32_t>(r);
}

__global__ __launch_bounds__(256) void k_inverse(const int32_t* __restrict__ perm, int64_t n,
                                                 int32_t* __restrict__ iperm) {
  const int64_t q = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (q < n) iperm[perm[q]] = static_cast<int32_t>(q);
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t* __restrict__ a, int32_t v, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t r = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; r < n; r += stride)
    a[r] = v;
}

// f = s layout: chunk_off[i] = first chunk of offset i's run (runs padded to
// whole chunks of kSegRows), hdrs[i].n_out = k_i, hdrs[K].n_out = padded length
__global__ void k_chunk_layout(const int64_t* __restrict__ pair_off, int K,
                               int32_t* __restrict__ chunk_off, DeviceHeader* __restrict__ hdrs) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int64_t c = 0;
  for (int i = 0; i < K; ++i) {
    const int64_t k_i = pair_off[i + 1] - pair_off[i];
    chunk_off[i] = static_cast<int32_t>(c);
    hdrs[i].status = 0;
    hdrs[i].n_out = k_i;
    c += (k_i + kSegRows - 1) / kSegRows;
  }
  chunk_off[K] = static_cast<int32_t>(c);
  hdrs[K].status = 0;
  hdrs[K].n_out = c * kSegRows;
}

// seg[c] = the offset whose run holds chunk c (0 past the last run)
__global__ __launch_bounds__(256) void k_seg_fill(const int32_t* __restrict__ chunk_off, int K,
                                                  int64_t nchunks, int32_t* __restrict__ seg) {
  const int64_t c = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (c >= nchunks) return;
  int lo = 0, hi = K;                 // chunk_off[lo] <= c < chunk_off[hi], else 0
  if (c >= chunk_off[K]) {
    seg[c] = 0;
    return;
  }
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (chunk_off[mid] <= c) lo = mid; else hi = mid;
  }
  seg[c] = lo;
}

// pair e of R_i -> position chunk_off[i] kSegRows + (e - pair_off[i]):
// src = 1 + SC output row, dst = SC input row
__global__ __launch_bounds__(256) void k_seg_scatter(const int32_t* __restrict__ pairs,
                                                     const int64_t* __restrict__ pair_off, int K,
                                                     const int32_t* __restrict__ chunk_off,
                                                     int32_t* __restrict__ src,
                                                     int32_t* __restrict__ dst) {
  const int64_t total = pair_off[K];
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += stride) {
    int lo = 0, hi = K;
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      if (pair_off[mid] <= e) lo = mid; else hi = mid;
    }
    const int64_t pos = static_cast<int64_t>(chunk_off[lo]) * kSegRows + (e - pair_off[lo]);
    src[pos] = pairs[2 * e + 1] + 1;
    dst[pos] = pairs[2 * e];
  }
}

__global__ void k_set_rows(DeviceHeader* h, int64_t n) {
  if (threadIdx.x == 0) {
    h->status = 0;
    h->n_out = n;
  }
}

// One lane per pair of the rule book (R_0 first); the pair's offset is found
// by a binary search of the offset table.
__global__ __launch_bounds__(256) void k_scatter_transpose(
    const int32_t* __restrict__ pairs, const int64_t* __restrict__ pair_off, int K,
    const int32_t* __restrict__ iperm, int32_t* __restrict__ tgmap, int64_t tgstride) {
  const int64_t total = pair_off[K];
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += stride) {
    int lo = 0, hi = K;            // pair_off[lo] <= e < pair_off[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      if (pair_off[mid] <= e) lo = mid; else hi = mid;
    }
    const int32_t a = pairs[2 * e], b = pairs[2 * e + 1];
    tgmap[lo * tgstride + iperm[a]] = b + 1;
  }
}

// ---------------------------------------------------------------------------
// Weight and bias gradients
// ---------------------------------------------------------------------------
constexpr int64_t kChunk = 4096;   // output positions (so at most as many pairs) per partial
constexpr int kSub = 64;           // pairs staged in LDS at a time

// The (offset, chunk) of this workgroup and its pair range inside R_i, from
// the rule book's per-block bases (blk_base[i][b] = first pair of R_i whose
// output is in block b of kBlock positions).  Workgroup L runs on XCD L mod 8;
// the K offsets of one chunk go to one XCD, so that the rows they share
// (every output row of the chunk, and its neighbours) meet in that L2.
struct DwChunk {
  int i, c;
  int64_t start, end;      // pair range [start, end) relative to R_i
};
__device__ __forceinline__ bool dw_chunk(const int32_t* blk_base, const int64_t* pair_off,
                                         int64_t nblk, int K, int nchunk, DwChunk* d) {
  const int L = blockIdx.x, xcd = L % 8, q = L / 8;
  d->c = xcd + 8 * (q / K);
  d->i = q % K;
  if (d->c >= nchunk) return false;
  constexpr int64_t kBpc = kChunk / kBlock;     // rule-book blocks per chunk
  const int64_t b0 = d->c * kBpc, b1 = b0 + kBpc;
  const int64_t k_i = pair_off[d->i + 1] - pair_off[d->i];
  d->start = blk_base[d->i * nblk + b0];
  d->end = b1 < nblk ? blk_base[d->i * nblk + b1] : k_i;
  return true;
}
constexpr int64_t kRowChunk = 512;    // rows per bias-gradient partial

// grid: (8 K ceil(nchunk / 8) (offset, chunk) pairs, see dw_chunk; tile);
// tile = (c-block of 64) x (n-block of 64).
template <typename T, bool DC>
__global__ __launch_bounds__(256) void k_dw_partial(
    const int32_t* __restrict__ pairs, const int64_t* __restrict__ pair_off,
    const int32_t* __restrict__ blk_base, int64_t nblk, const T* __restrict__ x,
    const T* __restrict__ dy, int C_in, int C_out, int K, int nchunk, float* __restrict__ part) {
  __shared__ float s_x[kSub][64 + 1];
  __shared__ float s_g[kSub][64 + 1];
  __shared__ int32_t s_a[kSub], s_b[kSub];
  DwChunk dc_;
  if (!dw_chunk(blk_base, pair_off, nblk, K, nchunk, &dc_)) return;
  const int i = dc_.i, chunk = dc_.c;
  const int ntn = (C_out + 63) / 64;
  const int c0 = (blockIdx.y / ntn) * 64, n0 = (blockIdx.y % ntn) * 64;
  const int64_t base = pair_off[i];
  const int64_t start = dc_.start, end = dc_.end;
  const int tc = threadIdx.x / 16, tn = threadIdx.x % 16;
  float acc[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[u][v] = 0.0f;
  for (int64_t sub = start; sub < end; sub += kSub) {
    const int np = static_cast<int>(end - sub < kSub ? end - sub : kSub);
    if (threadIdx.x < np) {
      const int32_t a = pairs[2 * (base + sub + threadIdx.x)];
      const int32_t b = pairs[2 * (base + sub + threadIdx.x) + 1];
      // (input row, gradient row): (a, b) for VSC / SC; DC reads its pairs backwards
      s_a[threadIdx.x] = DC ? b : a;
      s_b[threadIdx.x] = DC ? a : b;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kSub * 64; e += 256) {
      const int pp = e / 64, cc = e % 64;
      float xv = 0.0f, gv = 0.0f;
      if (pp < np) {
        if (c0 + cc < C_in) xv = IO<T>::ld(x, static_cast<int64_t>(s_a[pp]) * C_in + c0 + cc);
        if (n0 + cc < C_out) gv = IO<T>::ld(dy, static_cast<int64_t>(s_b[pp]) * C_out + n0 + cc);
      }
      s_x[pp][cc] = xv;
      s_g[pp][cc] = gv;
    }
    __syncthreads();
    for (int pp = 0; pp < np; ++pp) {
      float xr[4], gr[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) xr[u] = s_x[pp][tc * 4 + u];
#pragma unroll
      for (int v = 0; v < 4; ++v) gr[v] = s_g[pp][tn * 4 + v];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(xr[u], gr[v], acc[u][v]);
    }
    __syncthreads();
  }
  float* out = part + (static_cast<int64_t>(i) * nchunk + chunk) * C_in * C_out;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = c0 + tc * 4 + u;
    if (c >= C_in) continue;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int n = n0 + tn * 4 + v;
      if (n < C_out) out[static_cast<int64_t>(c) * C_out + n] = acc[u][v];
    }
  }
}

// Matrix-core partial products (bf16 inputs, fp32 accumulation): grid
// (chunk, offset, 64x64 tile of dW^i).  Per step 64 pairs: their input rows
// and gradient rows (this tile's 64 columns of each) are gathered into LDS
// row-major, 8 lanes per 128-byte row; wave w multiplies all pairs of the
// step, 32 at a time in order, into its own 32x32 quadrant of the tile (so
// each result is one in-order sum, written straight out, and a wave holds 16
// accumulator registers; with 64-pair steps four workgroups share a compute
// unit, which hides the gathers' latency better than larger steps with fewer
// workgroups).
// The contraction runs over pairs, so an operand fragment holds one channel
// of 8 consecutive pairs: it comes from the row-major tile through gfx950's
// transposing LDS read (16 lanes read 4 pairs x 16 channels, each lane
// receives one channel of the 4 pairs).  Columns past C_in / C_out are zero.
// dbpart != NULL (VSC): the workgroups of the centre offset, whose pairs are
// every output row once, also sum the gradient rows (the bias gradient) with
// two more products per 32 pairs, a fragment of ones times the staged rows,
// in waves 0 and 1 of the first channel tile; dbpart[chunk][n] receives the
// chunk's column sums.
typedef short dw_s4 __attribute__((ext_vector_type(4)));
typedef __bf16 dw_bf8 __attribute__((ext_vector_type(8)));
typedef float dw_f4 __attribute__((ext_vector_type(4)));
typedef unsigned dw_u4 __attribute__((ext_vector_type(4)));

// Tiles of 64-channel rows (128 bytes) in LDS store the 16-byte chunk k of
// row r at chunk k ^ (r & 7): the rows read together by one transposing read
// then fall on different banks (unswizzled 128-byte rows all start on the
// same bank).
__device__ __forceinline__ int dw_swz(int row, int col) {
  return row * 64 + ((((col >> 3) ^ (row & 7)) << 3) | (col & 7));
}

__device__ __forceinline__ dw_bf8 tr_frag(const uint16_t* tile, int p0, int c0, int lane) {
  // lanes 16q + j: pairs p0 + 8q + j/4 (+4 for the upper half), channels c0 + 4(j%4)..+3
  const int j = lane & 15, q = lane >> 4;
  const int row = p0 + 8 * q + (j >> 2), col = c0 + 4 * (j & 3);
  typedef __attribute__((address_space(3))) dw_s4 lds_s4;
  // generic -> LDS address-space conversion (the tile is a __shared__ array)
  lds_s4* lo = (lds_s4*)(const_cast<uint16_t*>(tile) + dw_swz(row, col));
  lds_s4* hi = (lds_s4*)(const_cast<uint16_t*>(tile) + dw_swz(row + 4, col));
  const dw_s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(lo);
  const dw_s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(hi);
  typedef short s8 __attribute__((ext_vector_type(8)));
  const s8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(dw_bf8, v);
}

template <bool DC>
__global__ __launch_bounds__(256, 4) void k_dw_mfma(
    const int32_t* __restrict__ pairs, const int64_t* __restrict__ pair_off,
    const int32_t* __restrict__ blk_base, int64_t nblk, const uint16_t* __restrict__ x,
    const uint16_t* __restrict__ dy, int C_in, int C_out, int K, int nchunk,
    float* __restrict__ part, int centre, float* __restrict__ dbpart) {
  constexpr int STEP = 64;
  constexpr int PASS = STEP / 32;                      // 32 rows per pass of 256 lanes
  // staging tiles and a ring of the pairs of four steps: 18 KB
  __shared__ __attribute__((aligned(16))) uint16_t s_buf[2 * STEP * 64];
  __shared__ int2 s_pr[4][STEP];
  uint16_t* s_x = s_buf;
  uint16_t* s_g = s_buf + STEP * 64;
  DwChunk dc_;
  if (!dw_chunk(blk_base, pair_off, nblk, K, nchunk, &dc_)) return;
  const int i = dc_.i, chunk = dc_.c;
  const int ntn = (C_out + 63) / 64;
  const int c0 = (blockIdx.y / ntn) * 64, n0 = (blockIdx.y % ntn) * 64;
  const int64_t base = pair_off[i];
  const int64_t start = dc_.start, end = dc_.end;
  const int nsteps = static_cast<int>((end - start + STEP - 1) / STEP);
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int cx = C_in - c0 < 64 ? C_in - c0 : 64;     // valid columns of this tile
  const int cg = C_out - n0 < 64 ? C_out - n0 : 64;
  float* out = part + (static_cast<int64_t>(i) * nchunk + chunk) * C_in * C_out;
  const bool dbt = dbpart && i == centre && c0 == 0;    // this tile sums the bias gradient
  if (nsteps == 0) {                                   // no pair of R_i in this chunk
    for (int t = threadIdx.x; t < 64 * 64; t += 256) {
      const int c = c0 + t / 64, n = n0 + t % 64;
      if (c < C_in && n < C_out) out[static_cast<int64_t>(c) * C_out + n] = 0.0f;
    }
    if (dbt && threadIdx.x < 64 && n0 + threadIdx.x < C_out)
      dbpart[static_cast<int64_t>(chunk) * C_out + n0 + threadIdx.x] = 0.0f;
    return;
  }

  // Over steps of STEP pairs: at step t the pairs of step t + 3 are loaded
  // (threads 0..STEP-1, one each) and, after the MFMAs, put in the LDS ring;
  // the data rows of step t + 2 are gathered (their pairs from the ring) into
  // one of two register sets, the MFMAs of step t run on the LDS tiles, and
  // the rows of step t + 1 (the other set) are written to LDS.  Every load is
  // unconditional (pairs past the chunk read its first pair; rows past the
  // chunk and columns past C read row 0 / column 0 and are zeroed when
  // staged), so no load sits under a branch, and the issue order (the pair
  // before the rows) lets the in-order load counter keep the rows in flight
  // while the pair is waited on.
  const int npairs = static_cast<int>(end - start);
  const int ch = (threadIdx.x % 8) * 8;                // this lane's 8 columns
  const bool colx = ch < cx, colg = ch < cg;
  typedef dw_u4 Rows[PASS];
  auto pair_load = [&](int t) __attribute__((always_inline)) -> int2 {
    const int e = t * STEP + (threadIdx.x < STEP ? threadIdx.x : 0);
    return *reinterpret_cast<const int2*>(pairs + 2 * (base + start + (e < npairs ? e : 0)));
  };
  auto pair_put = [&](int t, int2 v) __attribute__((always_inline)) {
    if (threadIdx.x < STEP) s_pr[t & 3][threadIdx.x] = v;
  };
  auto gather = [&](int t, Rows& vx, Rows& vg, uint32_t& ok) __attribute__((always_inline)) {
    ok = 0;
#pragma unroll
    for (int pass = 0; pass < PASS; ++pass) {
      const int e = t * STEP + pass * 32 + threadIdx.x / 8;
      const int2 pr = s_pr[t & 3][pass * 32 + threadIdx.x / 8];
      // (input row, gradient row); DC reads its pairs backwards
      const int32_t ra = DC ? pr.y : pr.x, rg = DC ? pr.x : pr.y;
      const bool okx = e < npairs && colx, okg = e < npairs && colg;
      ok |= (okx ? 1u : 0u) << (2 * pass) | (okg ? 2u : 0u) << (2 * pass);
      vx[pass] = *reinterpret_cast<const dw_u4*>(
          x + (okx ? static_cast<int64_t>(ra) * C_in + c0 + ch : 0));
      vg[pass] = *reinterpret_cast<const dw_u4*>(
          dy + (okg ? static_cast<int64_t>(rg) * C_out + n0 + ch : 0));
    }
  };
  auto stage = [&](const Rows& vx, const Rows& vg, uint32_t ok) __attribute__((always_inline)) {
    const dw_u4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int pass = 0; pass < PASS; ++pass) {
      const int pp = pass * 32 + threadIdx.x / 8;
      *reinterpret_cast<dw_u4*>(&s_x[dw_swz(pp, ch)]) = (ok >> (2 * pass)) & 1u ? vx[pass] : z;
      *reinterpret_cast<dw_u4*>(&s_g[dw_swz(pp, ch)]) = (ok >> (2 * pass)) & 2u ? vg[pass] : z;
    }
  };

  // wave w owns the 32 x 32 quadrant (channel blocks 2 (w / 2) + uu, gradient
  // blocks 2 (w % 2) + vv) of the 64 x 64 tile, over all pairs of the chunk
  const int ub = 2 * (wave / 2), vb = 2 * (wave % 2);
  dw_f4 acc[2][2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v) acc[u][v] = dw_f4{0.f, 0.f, 0.f, 0.f};
  const bool dbw = dbt && wave < 2;                    // waves 0, 1 cover all 4 column blocks
  dw_f4 accb[2] = {dw_f4{0.f, 0.f, 0.f, 0.f}, dw_f4{0.f, 0.f, 0.f, 0.f}};
  dw_bf8 ones;
#pragma unroll
  for (int k = 0; k < 8; ++k) ones[k] = static_cast<__bf16>(1.0f);

  Rows xa, ga, xb, gb;
  uint32_t oka = 0, okb = 0;
  pair_put(0, pair_load(0));
  pair_put(1, pair_load(1));
  pair_put(2, pair_load(2));
  __syncthreads();
  gather(0, xa, ga, oka);
  gather(1, xb, gb, okb);
  stage(xa, ga, oka);
  __syncthreads();
  // step t: the set holding step t + 1 is `nx`, the free set `fr`
  // (the gather of step t + 2 is issued even past the last step, as rows that
  // are all zeroed, so that the number of loads in flight never depends on t)
  auto step = [&](int t, Rows& nxx, Rows& nxg, uint32_t& nok, Rows& frx, Rows& frg,
                  uint32_t& fok) __attribute__((always_inline)) {
    const int2 pn = pair_load(t + 3);
    gather(t + 2, frx, frg, fok);
#pragma unroll
    for (int kc = 0; kc < STEP / 32; ++kc) {   // the step's pairs, 32 at a time, in order
      dw_bf8 fa[2], fb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) fa[u] = tr_frag(s_x, kc * 32, (ub + u) * 16, lane);
#pragma unroll
      for (int v = 0; v < 2; ++v) fb[v] = tr_frag(s_g, kc * 32, (vb + v) * 16, lane);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int v = 0; v < 2; ++v)
          acc[u][v] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[u], fb[v], acc[u][v], 0, 0, 0);
      if (dbw) {
#pragma unroll
        for (int v = 0; v < 2; ++v)
          accb[v] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, fb[v], accb[v], 0, 0, 0);
      }
    }
    __syncthreads();                           // tiles (and ring slot t + 3 = t - 1) free
    if (t + 1 < nsteps) stage(nxx, nxg, nok);
    pair_put(t + 3, pn);
    __syncthreads();
  };
  int t = 0;
  for (; t + 1 < nsteps; t += 2) {
    step(t, xb, gb, okb, xa, ga, oka);
    step(t + 1, xa, ga, oka, xb, gb, okb);
  }
  if (t < nsteps) step(t, xb, gb, okb, xa, ga, oka);
  // lane (r, g) holds rows 4g + e, column r of each 16x16 block
  const int r = lane % 16, g = lane / 16;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = c0 + (ub + u) * 16 + 4 * g + e, n = n0 + (vb + v) * 16 + r;
        if (c < C_in && n < C_out) out[static_cast<int64_t>(c) * C_out + n] = acc[u][v][e];
      }
  if (dbw && g == 0) {                                 // every row of accb holds the sums
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int n = n0 + (vb + v) * 16 + r;
      if (n < C_out) dbpart[static_cast<int64_t>(chunk) * C_out + n] = accb[v][0];
    }
  }
}

// Bias gradient, stage 2 (workgroups of k_dw_reduce past the weight's): 4
// columns per workgroup; lane (phase q of 64, column) adds chunk partials q,
// q + 64, ... eight loads at a time into 8 accumulators (by round), then the
// 64 phases are added in a fixed tree.
__device__ void db_reduce_block(const float* __restrict__ partb, int nchunks, int C_out,
                                float* __restrict__ db, int blk) {
  constexpr int kPh = 64, kCols = 4;
  __shared__ float s[kPh][kCols + 1];
  const int q = threadIdx.x / kCols, cn = threadIdx.x % kCols;
  const int n = blk * kCols + cn;
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (n < C_out) {
    int ch = q;
    for (; ch + 7 * kPh < nchunks; ch += 8 * kPh) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = partb[static_cast<int64_t>(ch + u * kPh) * C_out + n];
#pragma unroll
      for (int u = 0; u < 8; ++u) a[u] += v[u];
    }
    for (int u = 0; ch < nchunks; ch += kPh, ++u)
      a[u] += partb[static_cast<int64_t>(ch) * C_out + n];
  }
  s[q][cn] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  __syncthreads();
  for (int h = kPh / 2; h >= 1; h >>= 1) {
    if (q < h) s[q][cn] += s[q + h][cn];
    __syncthreads();
  }
  if (q == 0 && n < C_out) db[n] = s[0][cn];
}

// dw[i][c][n] = sum over the chunks of R_i.  The chunks are split into S
// consecutive segments (S = 1, 2, 4 or 8, chosen on the host so that small
// weight tensors still fill the device); in a segment chunk ch goes to
// accumulator ch mod 8 and the 8 accumulators are added in a fixed tree; the
// segments' sums are added in a fixed tree through LDS.  Every order is
// fixed, so the result is reproducible.  A workgroup covers 256 / S
// consecutive elements; its threads with the same segment read consecutive
// elements of a partial.  Workgroups from nb_dw on reduce the bias
// gradient's partials instead (db_reduce_block).
__global__ __launch_bounds__(256) void k_dw_reduce(const float* __restrict__ part, int K,
                                                   int C_in, int C_out, int nch, int S,
                                                   float* __restrict__ dw, int64_t nb_dw,
                                                   const float* __restrict__ partb, int nrc,
                                                   float* __restrict__ db) {
  if (blockIdx.x >= nb_dw) {
    db_reduce_block(partb, nrc, C_out, db, static_cast<int>(blockIdx.x - nb_dw));
    return;
  }
  __shared__ float s_seg[256];
  const int64_t per = static_cast<int64_t>(C_in) * C_out;
  const int E = 256 / S;                       // elements per workgroup
  const int el = threadIdx.x % E, seg = threadIdx.x / E;
  const int64_t idx = blockIdx.x * static_cast<int64_t>(E) + el;
  const bool live = idx < K * per;
  const int L = (nch + S - 1) / S;
  const int c0 = seg * L < nch ? seg * L : nch;
  const int c1 = c0 + L < nch ? c0 + L : nch;
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (live) {
    const int i = static_cast<int>(idx / per);
    const int64_t rem = idx - i * per;
    const float* p = part + static_cast<int64_t>(i) * nch * per + rem;
    int ch = c0;
    for (; ch + 8 <= c1; ch += 8) {
#pragma unroll
      for (int j = 0; j < 8; ++j) a[j] += p[static_cast<int64_t>(ch + j) * per];
    }
    for (int j = 0; ch + j < c1; ++j) a[j] += p[static_cast<int64_t>(ch + j) * per];
  }
  s_seg[threadIdx.x] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  __syncthreads();
  for (int h = S / 2; h >= 1; h /= 2) {        // segment t += segment t + h, t < h
    if (seg < h) s_seg[threadIdx.x] += s_seg[threadIdx.x + h * E];
    __syncthreads();
  }
  if (seg == 0 && live) dw[idx] = s_seg[threadIdx.x];
}

// Bias gradient, stage 1: a chunk of kRowChunk rows per workgroup and up to
// 32 groups of 16 bytes of columns (grid.y covers wider rows); lane (row
// phase ph, column group cg) sums rows ph, ph + P, ... of the chunk (P the
// largest power of two that fits, loads issued 8 rows at a time), then the
// phases are added in a fixed tree through LDS.
template <typename T>
__global__ __launch_bounds__(256) void k_db_partial(const T* __restrict__ dy, int64_t rows,
                                                    int C_out, float* __restrict__ partb) {
  constexpr int V = IO<T>::kVec;
  __shared__ float s[256][V + 1];
  const int ngrp_all = (C_out + V - 1) / V;       // 16-byte column groups of a row
  const int g0 = blockIdx.y * 32;
  const int ngrp = ngrp_all - g0 < 32 ? ngrp_all - g0 : 32;
  int nph = 1;
  while (nph * 2 * ngrp <= 256) nph *= 2;         // row phases: a power of two
  const int ph = threadIdx.x / ngrp, cgp = g0 + threadIdx.x % ngrp;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kRowChunk;
  const int64_t r1 = r0 + kRowChunk < rows ? r0 + kRowChunk : rows;
  float acc[V];
#pragma unroll
  for (int e = 0; e < V; ++e) acc[e] = 0.0f;
  const bool vec = C_out % V == 0;
  auto row_vals = [&](int64_t r, float* v) {
    if (vec) {
      IO<T>::ld16(dy, r * C_out + cgp * V, v);
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e)
        v[e] = cgp * V + e < C_out ? IO<T>::ld(dy, r * C_out + cgp * V + e) : 0.0f;
    }
  };
  if (ph < nph) {
    int64_t r = r0 + ph;
    for (; r + 7 * nph < r1; r += 8 * nph) {      // 8 rows in flight, added in row order
      float v[8][V];
#pragma unroll
      for (int u = 0; u < 8; ++u) row_vals(r + u * nph, v[u]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] += v[u][e];
    }
    for (; r < r1; r += nph) {
      float v[V];
      row_vals(r, v);
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e] += v[e];
    }
  }
#pragma unroll
  for (int e = 0; e < V; ++e) s[threadIdx.x][e] = acc[e];
  __syncthreads();
  for (int h = nph / 2; h >= 1; h >>= 1) {        // phase p absorbs phase p + h
    if (ph < h) {
#pragma unroll
      for (int e = 0; e < V; ++e) s[threadIdx.x][e] += s[threadIdx.x + h * ngrp][e];
    }
    __syncthreads();
  }
  if (ph == 0) {
#pragma unroll
    for (int e = 0; e < V; ++e) {
      const int n = cgp * V + e;
      if (n < C_out) partb[static_cast<int64_t>(blockIdx.x) * C_out + n] = s[threadIdx.x][e];
    }
  }
}


int64_t dw_nchunk(spconv_rulebook rb) {
  constexpr int64_t kBpc = kChunk / kBlock;
  return (rb->nblk + kBpc - 1) / kBpc;
}

}  // namespace

// ---------------------------------------------------------------------------
// Host entry points (called by abi.hip after argument checks)
// ---------------------------------------------------------------------------
int pool_forward(spconv_rulebook rb, int mode, int dt, const void* x, void* y, int C,
                 hipStream_t st) {
  if (rb->n_cap == 0) return SPCONV_OK;
  if (dt == SPCONV_F32) {
    if (mode == SPCONV_POOL_MAX) launch_pool<float, true>(rb, x, y, C, st);
    else launch_pool<float, false>(rb, x, y, C, st);
  } else {
    if (mode == SPCONV_POOL_MAX) launch_pool<uint16_t, true>(rb, x, y, C, st);
    else launch_pool<uint16_t, false>(rb, x, y, C, st);
  }
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

static int64_t seg_cap(int64_t n_in, int64_t K) { return n_in + K * kSegRows; }

size_t transpose_bytes(int64_t n_in, int64_t K) {
  const int64_t tgstride = ((n_in + kBlock - 1) / kBlock) * kBlock;
  const int64_t npad = seg_cap(n_in, K);
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  return al(256) + al(static_cast<size_t>(n_in) * 4) + al(static_cast<size_t>(K * tgstride) * 4) +
         2 * al(static_cast<size_t>(npad) * 4) + al(static_cast<size_t>(npad / kSegRows + 1) * 4) +
         al(static_cast<size_t>(K + 1) * 4) + al(static_cast<size_t>(K + 1) * sizeof(DeviceHeader));
}

int build_transpose(spconv_rulebook rb, const int32_t* coords, char* mem) {
  const int64_t n = rb->n_in;
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  rb->t_hdr = reinterpret_cast<DeviceHeader*>(mem);
  rb->t_perm = reinterpret_cast<int32_t*>(mem + al(256));
  rb->t_gstride = ((n + kBlock - 1) / kBlock) * kBlock;
  rb->t_gmap = reinterpret_cast<int32_t*>(mem + al(256) + al(static_cast<size_t>(n) * 4));
  {
    char* q = mem + al(256) + al(static_cast<size_t>(n) * 4) +
              al(static_cast<size_t>(rb->K * rb->t_gstride) * 4);
    rb->t_npad_cap = seg_cap(n, rb->K);
    const size_t pb = al(static_cast<size_t>(rb->t_npad_cap) * 4);
    rb->t_src = reinterpret_cast<int32_t*>(q);
    rb->t_dst = reinterpret_cast<int32_t*>(q + pb);
    rb->t_seg = reinterpret_cast<int32_t*>(q + 2 * pb);
    const size_t sb = al(static_cast<size_t>(rb->t_npad_cap / kSegRows + 1) * 4);
    rb->t_chunk_off = reinterpret_cast<int32_t*>(q + 2 * pb + sb);
    rb->t_hdrs = reinterpret_cast<DeviceHeader*>(q + 2 * pb + sb +
                                                 al(static_cast<size_t>(rb->K + 1) * 4));
  }
  rb->t_single = true;               // f = s: one pair per SC input row
  for (int j = 1; j < rb->D; ++j) rb->t_single = rb->t_single && rb->f[j] == rb->s[j];
  hipStream_t st = rb->stream;
  k_set_rows<<<1, 64, 0, st>>>(rb->t_hdr, n);
  k_fill_i32<<<grid_of(rb->K * rb->t_gstride), 256, 0, st>>>(rb->t_gmap, 0, rb->K * rb->t_gstride);
  if (n == 0) return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;

  ClassGeom g{};
  g.D = rb->D;
  int64_t classes = 1;
  for (int j = rb->D - 1; j >= 1; --j) {
    g.s[j] = rb->s[j];
    g.mult[j] = classes;
    classes *= rb->s[j];
  }
  const size_t scratch = radix_sort_scratch_bytes(n);
  const size_t tbytes = 2 * al(static_cast<size_t>(n) * 8) + 3 * al(static_cast<size_t>(n) * 4) +
                        al(scratch);
  void* tmem = nullptr;
  if (dev_alloc(rb, tbytes, st, &tmem) != SPCONV_OK) return SPCONV_ENOMEM;
  char* p = static_cast<char*>(tmem);
  uint64_t* keys = reinterpret_cast<uint64_t*>(p);
  uint64_t* keys_tmp = reinterpret_cast<uint64_t*>(p + al(n * 8));
  int32_t* vals = reinterpret_cast<int32_t*>(p + 2 * al(n * 8));
  int32_t* vals_tmp = reinterpret_cast<int32_t*>(p + 2 * al(n * 8) + al(n * 4));
  int32_t* iperm = reinterpret_cast<int32_t*>(p + 2 * al(n * 8) + 2 * al(n * 4));
  void* sort_scratch = p + 2 * al(n * 8) + 3 * al(n * 4);
  if (classes > 1) {
    k_class_keys<<<grid_of(n, 1ll << 30), 256, 0, st>>>(coords, n, g, keys, vals);
    const bool flipped = radix_sort_pairs(keys, vals, keys_tmp, vals_tmp, rb->t_hdr, n,
                                          bitlen(static_cast<uint64_t>(classes - 1)), sort_scratch,
                                          st);
    if (hipMemcpyAsync(rb->t_perm, flipped ? vals_tmp : vals, static_cast<size_t>(n) * 4,
                       hipMemcpyDeviceToDevice, st) != hipSuccess) {
      (void)hipGetLastError();
      (void)dev_free(rb, tmem, st);
      return SPCONV_EHIP;
    }
  } else {
    k_iota<<<grid_of(n, 1ll << 30), 256, 0, st>>>(rb->t_perm, n);
  }
  k_inverse<<<grid_of(n, 1ll << 30), 256, 0, st>>>(rb->t_perm, n, iperm);
  k_scatter_transpose<<<grid_of(rb->K * n), 256, 0, st>>>(rb->pairs, rb->pair_off,
                                                          static_cast<int>(rb->K), iperm,
                                                          rb->t_gmap, rb->t_gstride);
  if (rb->t_single) {
    const int64_t nchunks = rb->t_npad_cap / kSegRows + 1;
    k_fill_i32<<<grid_of(rb->t_npad_cap), 256, 0, st>>>(rb->t_src, 0, rb->t_npad_cap);
    k_fill_i32<<<grid_of(rb->t_npad_cap), 256, 0, st>>>(rb->t_dst, -1, rb->t_npad_cap);
    k_chunk_layout<<<1, 64, 0, st>>>(rb->pair_off, static_cast<int>(rb->K), rb->t_chunk_off,
                                     rb->t_hdrs);
    k_seg_fill<<<grid_of(nchunks, 1ll << 30), 256, 0, st>>>(rb->t_chunk_off,
                                                            static_cast<int>(rb->K), nchunks,
                                                            rb->t_seg);
    k_seg_scatter<<<grid_of(n), 256, 0, st>>>(rb->pairs, rb->pair_off, static_cast<int>(rb->K),
                                              rb->t_chunk_off, rb->t_src, rb->t_dst);
  }
  if (dev_free(rb, tmem, st) != SPCONV_OK) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

// The transposed direction with f = s: one single-offset launch per R_i
// (source rows pairs[.][1], destination rows pairs[.][0]), W^i sliced out of
// w.  Needs the offsets' lengths on the host (the rule book is synchronised
// once for that).  Returns kNotSingle, having launched nothing, when some
// SC input row has no pair.
int transpose_single(spconv_rulebook rb, int wmode, int in_dt, const void* x, const void* w,
                     const float* bias, int out_dt, void* y, int C_in, int C_out,
                     hipStream_t st) {
  if (rb->h_pair_off.empty()) {
    rb->h_pair_off.assign(static_cast<size_t>(rb->K + 1), 0);
    if (hipMemcpyAsync(rb->h_pair_off.data(), rb->pair_off, (rb->K + 1) * sizeof(int64_t),
                       hipMemcpyDeviceToHost, rb->stream) != hipSuccess ||
        hipStreamSynchronize(rb->stream) != hipSuccess) {
      (void)hipGetLastError();
      rb->h_pair_off.clear();
      return SPCONV_EHIP;
    }
  }
  // rows near the far border may lack a pair (their output site falls off
  // the SC grid); then not every destination row is written here
  if (rb->h_pair_off[rb->K] != rb->n_in) return kNotSingle;
  // one launch over all offsets when a matrix-core kernel fits the shape
  FwdView sv;
  sv.gmap = rb->t_src;
  sv.perm = rb->t_dst;
  sv.gstride = rb->t_npad_cap;
  sv.hdr = rb->t_hdrs + rb->K;
  sv.n_cap = rb->t_npad_cap;
  sv.K = 1;
  sv.n_src = rb->n_cap;
  sv.seg = rb->t_seg;
  const int r0 = forward_view(sv, wmode, in_dt, x, w, bias, out_dt, y, C_in, C_out, st);
  if (r0 != kNotSingle) return r0;
  // otherwise one launch per offset
  const size_t esz = in_dt == SPCONV_BF16 ? 2 : 4;
  int64_t chunk = 0;
  for (int64_t i = 0; i < rb->K; ++i) {
    const int64_t off = chunk * kSegRows, k_i = rb->h_pair_off[i + 1] - rb->h_pair_off[i];
    chunk += (k_i + kSegRows - 1) / kSegRows;
    if (k_i == 0) continue;
    FwdView v;
    v.gmap = rb->t_src + off;
    v.perm = rb->t_dst + off;
    v.gstride = k_i;
    v.hdr = rb->t_hdrs + i;
    v.n_cap = k_i;
    v.K = 1;
    v.n_src = rb->n_cap;
    v.seg = nullptr;
    const void* wi = static_cast<const char*>(w) + static_cast<size_t>(i) * C_in * C_out * esz;
    const int r = forward_view(v, wmode, in_dt, x, wi, bias, out_dt, y, C_in, C_out, st);
    if (r != SPCONV_OK) return r;
  }
  return SPCONV_OK;
}

FwdView transpose_view(spconv_rulebook rb) {
  FwdView v;
  v.gmap = rb->t_gmap;
  v.perm = rb->t_perm;
  v.gstride = rb->t_gstride;
  v.hdr = rb->t_hdr;
  v.n_cap = rb->n_in;
  v.K = rb->K;
  v.n_src = rb->n_cap;
  v.seg = nullptr;
  return v;
}

size_t backward_weight_workspace(spconv_rulebook rb, int C_in, int C_out, int op) {
  const int64_t rows = op == SPCONV_OP_DC ? rb->n_in : rb->n_cap;
  const int64_t nrc = (rows + kRowChunk - 1) / kRowChunk;
  return static_cast<size_t>(rb->K * dw_nchunk(rb)) * C_in * C_out * 4 +
         static_cast<size_t>(nrc > 0 ? nrc : 1) * C_out * 4 + 256;  // nrc >= the chunk count
}

int backward_weight(spconv_rulebook rb, int op, int dt, const void* x, const void* dy, float* dw,
                    float* db, int C_in, int C_out, void* ws, hipStream_t st) {
  const int nchunk = static_cast<int>(dw_nchunk(rb));
  const int K = static_cast<int>(rb->K);
  float* part = static_cast<float*>(ws);
  const int64_t per = static_cast<int64_t>(C_in) * C_out;
  // VSC on the matrix cores: the bias gradient comes from the weight
  // gradient's centre-offset workgroups (its pairs are every output row once,
  // each with itself), per chunk, into the bias partials' area (at least
  // nchunk rows of C_out floats)
  int centre = 0;
  for (int j = 0; j < rb->D; ++j) centre = centre * rb->f[j] + (rb->f[j] - 1) / 2;
  const bool db_fused = db && op == SPCONV_OP_VSC && nchunk > 0 && dt == SPCONV_BF16 &&
                        C_in % 8 == 0 && C_out % 8 == 0;
  float* partb_fused = part + static_cast<int64_t>(rb->K) * nchunk * per;
  if (nchunk > 0) {
    const int tiles = ((C_in + 63) / 64) * ((C_out + 63) / 64);
    // (offset, chunk) pairs: 8 XCDs x K offsets x ceil(nchunk / 8) chunks each
    dim3 grid(static_cast<unsigned>(8 * K * ((nchunk + 7) / 8)), static_cast<unsigned>(tiles));
    const bool dc = op == SPCONV_OP_DC;
    // matrix cores for bf16 rows of whole 16-byte chunks (C % 8 == 0 keeps
    // every gathered 16-byte load inside its row)
    if (dt == SPCONV_BF16 && C_in % 8 == 0 && C_out % 8 == 0) {
      auto kern = dc ? k_dw_mfma<true> : k_dw_mfma<false>;
      kern<<<grid, 256, 0, st>>>(rb->pairs, rb->pair_off, rb->blk_cnt, rb->nblk,
                                 static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(dy),
                                 C_in, C_out, K, nchunk, part, db_fused ? centre : -1,
                                 db_fused ? partb_fused : nullptr);
    } else if (dt == SPCONV_F32) {
      auto kern = dc ? k_dw_partial<float, true> : k_dw_partial<float, false>;
      kern<<<grid, 256, 0, st>>>(rb->pairs, rb->pair_off, rb->blk_cnt, rb->nblk,
                                 static_cast<const float*>(x), static_cast<const float*>(dy), C_in,
                                 C_out, K, nchunk, part);
    } else {
      auto kern = dc ? k_dw_partial<uint16_t, true> : k_dw_partial<uint16_t, false>;
      kern<<<grid, 256, 0, st>>>(rb->pairs, rb->pair_off, rb->blk_cnt, rb->nblk,
                                 static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(dy),
                                 C_in, C_out, K, nchunk, part);
    }
  }
  // bias-gradient partials: from k_dw_mfma (fused) or one pass over dy
  const float* partb = nullptr;
  int nrc = 0;
  if (db_fused) {
    partb = partb_fused;
    nrc = static_cast<int>(nchunk);
  } else if (db) {
    const int64_t rows = op == SPCONV_OP_DC ? rb->n_in : rb->n_out;
    nrc = static_cast<int>((rows + kRowChunk - 1) / kRowChunk);
    float* pb = part + static_cast<int64_t>(rb->K) * nchunk * per;
    partb = pb;
    if (nrc > 0) {
      const int vec = dt == SPCONV_F32 ? 4 : 8;
      const int groups = (C_out + vec - 1) / vec;
      dim3 g(static_cast<unsigned>(nrc), static_cast<unsigned>((groups + 31) / 32));
      if (dt == SPCONV_F32)
        k_db_partial<float><<<g, 256, 0, st>>>(static_cast<const float*>(dy), rows, C_out, pb);
      else
        k_db_partial<uint16_t><<<g, 256, 0, st>>>(static_cast<const uint16_t*>(dy), rows, C_out,
                                                  pb);
    }
  }
  {
    // one launch sums both: the weight's elements, then the bias columns.
    // Segments per weight element: enough threads for the device (~128 K),
    // at least 8 chunks per segment (more segments did not speed up the
    // headline's 95 MB of partials)
    const int64_t elems = static_cast<int64_t>(rb->K) * per;
    int S = 1;
    while (S < 8 && elems * S < (int64_t{1} << 17) && nchunk / (2 * S) >= 8) S *= 2;
    const int64_t E = 256 / S;
    const int64_t nb_dw = (elems + E - 1) / E;
    const int64_t nb_db = db ? (C_out + 3) / 4 : 0;
    if (nb_dw + nb_db > 0)
      k_dw_reduce<<<static_cast<unsigned>(nb_dw + nb_db), 256, 0, st>>>(
          part, K, C_in, C_out, nchunk, S, dw, nb_dw, partb, nrc, db);
  }
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

}  // namespace spc
