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
// over this map.
//
// Weight gradient dW^i = sum over the pairs of R_i of (input row)^T x (output
// gradient row): R_i is cut into chunks of kChunk pairs; one workgroup forms
// the fp32 partial product of a chunk for a 64x64 tile of dW^i (pairs staged
// in LDS, 4x4 outputs per lane, pairs in list order), and a second kernel
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
template <typename T, int VEC, bool MAX>
__global__ __launch_bounds__(256) void k_pool(const int32_t* __restrict__ gmap,
                                              const int32_t* __restrict__ perm, int64_t gstride,
                                              const DeviceHeader* __restrict__ hdr, int K,
                                              const T* __restrict__ x, T* __restrict__ y, int C) {
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
    for (int i = 0; i < K; ++i) {
      const int32_t g = gmap[i * gstride + p] - 1;
      if (g < 0) continue;
      float v[VEC];
      const int64_t base = static_cast<int64_t>(g) * C + c0;
      if constexpr (VEC == 1) {
        v[0] = IO<T>::ld(x, base);
      } else {
        IO<T>::ld16(x, base, v);
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = MAX ? fmaxf(acc[e], v[e]) : acc[e] + v[e];
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
constexpr int64_t kChunk = 4096;   // pairs per partial product
constexpr int kSub = 64;           // pairs staged in LDS at a time
constexpr int64_t kRowChunk = 4096;

// grid: (chunk, offset, tile); tile = (c-block of 64) x (n-block of 64).
template <typename T, bool DC>
__global__ __launch_bounds__(256) void k_dw_partial(
    const int32_t* __restrict__ pairs, const int64_t* __restrict__ pair_off,
    const T* __restrict__ x, const T* __restrict__ dy, int C_in, int C_out, int maxchunks,
    float* __restrict__ part) {
  __shared__ float s_x[kSub][64 + 1];
  __shared__ float s_g[kSub][64 + 1];
  __shared__ int32_t s_a[kSub], s_b[kSub];
  const int i = blockIdx.y, chunk = blockIdx.x;
  const int ntn = (C_out + 63) / 64;
  const int c0 = (blockIdx.z / ntn) * 64, n0 = (blockIdx.z % ntn) * 64;
  const int64_t base = pair_off[i];
  const int64_t k_i = pair_off[i + 1] - base;
  const int64_t start = static_cast<int64_t>(chunk) * kChunk;
  if (start >= k_i) return;
  const int64_t end = start + kChunk < k_i ? start + kChunk : k_i;
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
  float* out = part + (static_cast<int64_t>(i) * maxchunks + chunk) * C_in * C_out;
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

// dw[i][c][n] = sum over the chunks of R_i, in ascending chunk order.
__global__ __launch_bounds__(256) void k_dw_reduce(const float* __restrict__ part,
                                                   const int64_t* __restrict__ pair_off, int K,
                                                   int C_in, int C_out, int maxchunks,
                                                   float* __restrict__ dw) {
  const int64_t per = static_cast<int64_t>(C_in) * C_out;
  const int64_t idx = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (idx >= K * per) return;
  const int i = static_cast<int>(idx / per);
  const int64_t rem = idx - i * per;
  const int64_t k_i = pair_off[i + 1] - pair_off[i];
  const int nch = static_cast<int>((k_i + kChunk - 1) / kChunk);
  float s = 0.0f;
  const float* p = part + static_cast<int64_t>(i) * maxchunks * per + rem;
  for (int ch = 0; ch < nch; ++ch) s += p[static_cast<int64_t>(ch) * per];
  dw[idx] = s;
}

// Bias gradient, stage 1: per chunk of kRowChunk rows, 4 row phases x 64
// columns per workgroup, phases combined in LDS in fixed order.
template <typename T>
__global__ __launch_bounds__(256) void k_db_partial(const T* __restrict__ dy, int64_t rows,
                                                    int C_out, float* __restrict__ partb) {
  __shared__ float s[4][64];
  const int chunk = blockIdx.x, nb = blockIdx.y * 64;
  const int ph = threadIdx.x / 64, n = nb + threadIdx.x % 64;
  const int64_t r0 = static_cast<int64_t>(chunk) * kRowChunk;
  const int64_t r1 = r0 + kRowChunk < rows ? r0 + kRowChunk : rows;
  float acc = 0.0f;
  if (n < C_out)
    for (int64_t r = r0 + ph; r < r1; r += 4) acc += IO<T>::ld(dy, r * C_out + n);
  s[ph][threadIdx.x % 64] = acc;
  __syncthreads();
  if (ph == 0 && n < C_out)
    partb[static_cast<int64_t>(chunk) * C_out + n] =
        ((s[0][threadIdx.x] + s[1][threadIdx.x]) + s[2][threadIdx.x]) + s[3][threadIdx.x];
}

__global__ __launch_bounds__(256) void k_db_reduce(const float* __restrict__ partb, int nchunks,
                                                   int C_out, float* __restrict__ db) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= C_out) return;
  float s = 0.0f;
  for (int ch = 0; ch < nchunks; ++ch) s += partb[static_cast<int64_t>(ch) * C_out + n];
  db[n] = s;
}

int64_t dw_maxchunks(spconv_rulebook rb) { return (rb->n_cap + kChunk - 1) / kChunk; }

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

size_t transpose_bytes(int64_t n_in, int64_t K) {
  const int64_t tgstride = ((n_in + kBlock - 1) / kBlock) * kBlock;
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  return al(256) + al(static_cast<size_t>(n_in) * 4) + al(static_cast<size_t>(K * tgstride) * 4);
}

int build_transpose(spconv_rulebook rb, const int32_t* coords, char* mem) {
  const int64_t n = rb->n_in;
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  rb->t_hdr = reinterpret_cast<DeviceHeader*>(mem);
  rb->t_perm = reinterpret_cast<int32_t*>(mem + al(256));
  rb->t_gstride = ((n + kBlock - 1) / kBlock) * kBlock;
  rb->t_gmap = reinterpret_cast<int32_t*>(mem + al(256) + al(static_cast<size_t>(n) * 4));
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
  if (hipMallocAsync(&tmem, tbytes, st) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_ENOMEM;
  }
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
      (void)hipFreeAsync(tmem, st);
      return SPCONV_EHIP;
    }
  } else {
    k_iota<<<grid_of(n, 1ll << 30), 256, 0, st>>>(rb->t_perm, n);
  }
  k_inverse<<<grid_of(n, 1ll << 30), 256, 0, st>>>(rb->t_perm, n, iperm);
  k_scatter_transpose<<<grid_of(rb->K * n), 256, 0, st>>>(rb->pairs, rb->pair_off,
                                                          static_cast<int>(rb->K), iperm,
                                                          rb->t_gmap, rb->t_gstride);
  if (hipFreeAsync(tmem, st) != hipSuccess) return SPCONV_EHIP;
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
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
  return v;
}

size_t backward_weight_workspace(spconv_rulebook rb, int C_in, int C_out, int op) {
  const int64_t rows = op == SPCONV_OP_DC ? rb->n_in : rb->n_cap;
  const int64_t nrc = (rows + kRowChunk - 1) / kRowChunk;
  return static_cast<size_t>(rb->K * dw_maxchunks(rb)) * C_in * C_out * 4 +
         static_cast<size_t>(nrc > 0 ? nrc : 1) * C_out * 4 + 256;
}

int backward_weight(spconv_rulebook rb, int op, int dt, const void* x, const void* dy, float* dw,
                    float* db, int C_in, int C_out, void* ws, hipStream_t st) {
  const int maxchunks = static_cast<int>(dw_maxchunks(rb));
  float* part = static_cast<float*>(ws);
  const int64_t per = static_cast<int64_t>(C_in) * C_out;
  if (maxchunks > 0) {
    const int tiles = ((C_in + 63) / 64) * ((C_out + 63) / 64);
    dim3 grid(static_cast<unsigned>(maxchunks), static_cast<unsigned>(rb->K),
              static_cast<unsigned>(tiles));
    const bool dc = op == SPCONV_OP_DC;
    if (dt == SPCONV_F32) {
      auto kern = dc ? k_dw_partial<float, true> : k_dw_partial<float, false>;
      kern<<<grid, 256, 0, st>>>(rb->pairs, rb->pair_off, static_cast<const float*>(x),
                                 static_cast<const float*>(dy), C_in, C_out, maxchunks, part);
    } else {
      auto kern = dc ? k_dw_partial<uint16_t, true> : k_dw_partial<uint16_t, false>;
      kern<<<grid, 256, 0, st>>>(rb->pairs, rb->pair_off, static_cast<const uint16_t*>(x),
                                 static_cast<const uint16_t*>(dy), C_in, C_out, maxchunks, part);
    }
  }
  k_dw_reduce<<<grid_of(rb->K * per, 1ll << 30), 256, 0, st>>>(part, rb->pair_off,
                                                               static_cast<int>(rb->K), C_in,
                                                               C_out, maxchunks, dw);
  if (db) {
    const int64_t rows = op == SPCONV_OP_DC ? rb->n_in : rb->n_out;
    const int nrc = static_cast<int>((rows + kRowChunk - 1) / kRowChunk);
    float* partb = part + static_cast<int64_t>(rb->K) * maxchunks * per;
    if (nrc > 0) {
      dim3 g(static_cast<unsigned>(nrc), static_cast<unsigned>((C_out + 63) / 64));
      if (dt == SPCONV_F32)
        k_db_partial<float><<<g, 256, 0, st>>>(static_cast<const float*>(dy), rows, C_out, partb);
      else
        k_db_partial<uint16_t><<<g, 256, 0, st>>>(static_cast<const uint16_t*>(dy), rows, C_out,
                                                  partb);
    }
    k_db_reduce<<<grid_of(C_out), 256, 0, st>>>(partb, nrc, C_out, db);
  }
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

}  // namespace spc
