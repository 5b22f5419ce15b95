// Forward multiply-add kernels of SC / VSC on gfx950 (Section 4 of the paper: zero
// the output, then for every offset i and pair j add input row R_i(j,1)
// times W^i into output row R_i(j,2); Table 1: a*m*n multiply-adds per active
// output site).
//
// The kernels are output-stationary: a workgroup owns a tile of output rows
// (consecutive positions of the rule book's Z-order schedule, so the tile is
// spatially compact) and keeps their fp32 accumulators in registers while it
// walks the offsets in ascending order.  For offset i it gathers the input
// rows G[i][p] of its positions (the gather map built with the rule book;
// 1 + input row, 0 = no active input, read as zeros) and multiplies them by
// W^i.  Every output element is written once, by one lane, after a
// fixed-order sum: no atomics, bitwise reproducible.
//
//   k_fwd_mfma  dense contraction on the matrix cores: v_mfma 16x16x32 bf16
//               or 16x16x4 f32.  W^i is staged into LDS transposed (one row
//               per output column, XOR-swizzled chunks) and double-buffered
//               across offsets; gathered rows go straight from memory to
//               registers through buffer loads whose hardware range check
//               returns zero for absent neighbours; a 16-row block whose 16
//               rows all lack offset i skips its MFMAs (and, for filters
//               other than 3^3, its gathers).
//   k_fwd_lowc  at most 4 input planes (e.g. the 1 plane of a pen-stroke
//               input): one lane per (output row, 16 output columns), fp32
//               FMA chains, weights through the scalar cache.
//   k_fwd_vec   any other channel count: one lane per (output row, output
//               column), fp32 FMA chain.
#pragma once

#include <cstdlib>
#include <cstring>

#include "internal.h"

namespace spc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Test knob: SPCONV_FORCE_PATH=vec runs the vector path for shapes the
// matrix-core kernel covers.
bool force_vector_path() {
  const char* e = std::getenv("SPCONV_FORCE_PATH");
  return e && std::strcmp(e, "vec") == 0;
}

constexpr uint32_t kBufDword3 = 0x00020000u;   // gfx9 raw buffer descriptor word 3

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T> struct ElemIO;
template <> struct ElemIO<float> {
  __device__ static float load(const float* p, int64_t i) { return p[i]; }
  __device__ static void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct ElemIO<uint16_t> {
  __device__ static float load(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  __device__ static void store(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
};

// Buffer loads whose hardware range check returns zero for an offset past
// the resource (kBufOOB and up): a load that may have nothing to read needs
// no branch (a load under a branch forces a wait for every load in flight).
constexpr uint32_t kBufOOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes),
                                           static_cast<int>(kBufDword3));
}
template <typename T> struct BufIO;
template <> struct BufIO<float> {
  static constexpr uint32_t kSize = 4;
  __device__ static float load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
  }
};
template <> struct BufIO<uint16_t> {
  static constexpr uint32_t kSize = 2;
  __device__ static float load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
  }
};
// Gather-map entries of offsets i0 .. i0 + KB - 1 at position p, minus one
// (-1: no neighbour, or offset past K).
template <int KB>
__device__ __forceinline__ void load_map(const int32_t* gmap, int64_t gstride, int K, int i0,
                                         int64_t p, int32_t (&g)[KB]) {
  const uint32_t bytes = static_cast<uint32_t>(gstride * 4);
#pragma unroll
  for (int b = 0; b < KB; ++b) {
    const int i = i0 + b < K ? i0 + b : 0;
    const __amdgpu_buffer_rsrc_t r = buf_rsrc(gmap + static_cast<int64_t>(i) * gstride, bytes);
    const uint32_t off = i0 + b < K ? static_cast<uint32_t>(p) * 4u : kBufOOB;
    g[b] = static_cast<int32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0)) - 1;
  }
}

// ---------------------------------------------------------------------------
// Generic (vector ALU) path
// ---------------------------------------------------------------------------
// Weight modes: the multiply-add uses Wk^i (C_in x C_out of the kernel) =
//   WT 0: w[i]                     (w is [K][C_in][C_out], the forward)
//   WT 2: w[i]^T                   (w is [K][C_out][C_in]: the input gradient of
//                                   SC / DC, run over the reversed pairs)
//   WT 1: w[K-1-i]^T               (the input gradient of VSC: its pairs are
//                                   symmetric, (a,b) in R_i iff (b,a) in R_{K-1-i})
template <int WT>
__device__ __forceinline__ int64_t w_index(int i, int K, int c, int n, int C_in, int C_out) {
  if constexpr (WT == 0) return (static_cast<int64_t>(i) * C_in + c) * C_out + n;
  const int iw = WT == 1 ? K - 1 - i : i;
  return (static_cast<int64_t>(iw) * C_out + n) * C_in + c;
}

// Positions run over the capacity n_cap (known on the host) so that the
// loads of the gather map do not wait for the device-side row count; a
// position at or past the count contributes nothing and stores nothing.
// The map entries of 8 offsets are loaded together (and, for one input
// plane, their input values and weights), then accumulated in offset order.
template <typename TIn, typename TOut, int WT>
__global__ __launch_bounds__(256) void k_fwd_vec(
    const int32_t* __restrict__ gmap, const int32_t* __restrict__ perm, int64_t gstride,
    int64_t n_cap, const DeviceHeader* __restrict__ hdr, int K, const TIn* __restrict__ x,
    const TIn* __restrict__ w, const float* __restrict__ bias, TOut* __restrict__ y, int C_in,
    int C_out, Epilogue epi) {
  constexpr int KB = 8;
  const int64_t n_rows = hdr->n_out;
  const int64_t total = n_cap * C_out;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t idx = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; idx < total;
       idx += stride) {
    const int64_t p = idx / C_out;                 // schedule position
    const int col = static_cast<int>(idx - p * C_out);
    const bool live = p < n_rows;
    float acc = 0.0f;
    for (int i0 = 0; i0 < K; i0 += KB) {
      int32_t g[KB];
#pragma unroll
      for (int b = 0; b < KB; ++b) {          // in bounds for every b: no branch
        const int i = i0 + b < K ? i0 + b : K - 1;
        g[b] = gmap[static_cast<int64_t>(i) * gstride + p] - 1;
      }
#pragma unroll
      for (int b = 0; b < KB; ++b) g[b] = (live && i0 + b < K) ? g[b] : -1;
      if (C_in == 1) {
        float xv[KB], wv[KB];
#pragma unroll
        for (int b = 0; b < KB; ++b) {
          xv[b] = g[b] >= 0 ? ElemIO<TIn>::load(x, g[b]) : 0.0f;
          wv[b] = i0 + b < K ? ElemIO<TIn>::load(w, w_index<WT>(i0 + b, K, 0, col, 1, C_out))
                             : 0.0f;
        }
#pragma unroll
        for (int b = 0; b < KB; ++b)
          if (g[b] >= 0) acc = fmaf(xv[b], wv[b], acc);
      } else {
#pragma unroll
        for (int b = 0; b < KB; ++b) {
          if (g[b] < 0) continue;
          const int64_t xb = static_cast<int64_t>(g[b]) * C_in;
          for (int c = 0; c < C_in; ++c)
            acc = fmaf(ElemIO<TIn>::load(x, xb + c),
                       ElemIO<TIn>::load(w, w_index<WT>(i0 + b, K, c, col, C_in, C_out)), acc);
        }
      }
    }
    if (!live) continue;
    const int64_t o = static_cast<int64_t>(perm[p]) * C_out + col;
    if (epi.scale)
      acc = fmaf(acc, epi.scale[col], bias ? bias[col] : 0.0f);
    else if (bias)
      acc += bias[col];
    if (epi.res) acc += ElemIO<TOut>::load(static_cast<const TOut*>(epi.res), o);
    if (epi.relu) acc = acc < 0.0f ? 0.0f : acc;
    ElemIO<TOut>::store(y, o, acc);
  }
}

template <typename TOut, int NCB> struct OutStore;
template <int NCB> struct OutStore<float, NCB> {
  __device__ static void store(float* p, const float* v) {
    if constexpr (NCB == 4) {
      *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    } else if constexpr (NCB == 2) {
      *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
    } else {
      p[0] = v[0];
    }
  }
};
template <int NCB> struct OutStore<uint16_t, NCB> {
  __device__ static void store(uint16_t* p, const float* v) {
    if constexpr (NCB == 4) {
      uint2 u;
      u.x = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
      u.y = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
      *reinterpret_cast<uint2*>(p) = u;
    } else if constexpr (NCB == 2) {
      *reinterpret_cast<uint32_t*>(p) =
          f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
    } else {
      p[0] = f32_to_bf16(v[0]);
    }
  }
};

// NCB adjacent output elements as fp32 (the residual of the epilogue).
template <typename TOut, int NCB> struct OutLoad;
template <int NCB> struct OutLoad<float, NCB> {
  __device__ static void load(const float* p, float* v) {
    if constexpr (NCB == 4) {
      const float4 u = *reinterpret_cast<const float4*>(p);
      v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
    } else if constexpr (NCB == 2) {
      const float2 u = *reinterpret_cast<const float2*>(p);
      v[0] = u.x; v[1] = u.y;
    } else {
      v[0] = p[0];
    }
  }
};
template <int NCB> struct OutLoad<uint16_t, NCB> {
  __device__ static void load(const uint16_t* p, float* v) {
    if constexpr (NCB == 4) {
      const uint2 u = *reinterpret_cast<const uint2*>(p);
      v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
      v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
    } else if constexpr (NCB == 2) {
      const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
      v[0] = __uint_as_float(u << 16); v[1] = __uint_as_float(u & 0xffff0000u);
    } else {
      v[0] = bf16_to_f32(p[0]);
    }
  }
};

// Few input planes (C_in <= kLowCin, C_out a multiple of kLowCols): one
// thread per output position and kLowCols output columns, a block of threads
// on one column group.  The gather-map entries and input values of KB
// offsets at a time (9, or 16 for larger filters) are loaded together into
// registers; meanwhile the block stages those offsets' weights of its
// columns in LDS, which every lane then reads at the same address (a
// broadcast).  The finished rows go
// through LDS once more, so that each store instruction writes whole 16-byte
// pieces of few rows (4 lanes per row) instead of one element of 64 rows
// (on 476,000 pen-stroke rows, 1 -> 32 fp32: 40 us against 87 us; 32
// columns per thread instead of 16 took 106 us).  Same per-element summation
// order as k_fwd_vec.
constexpr int kLowCin = 4;
constexpr int kLowCols = 16;
template <typename TIn, typename TOut, int WT, int KB>
__global__ __launch_bounds__(256) void k_fwd_lowc(
    const int32_t* __restrict__ gmap, const int32_t* __restrict__ perm, int64_t gstride,
    int64_t n_cap, const DeviceHeader* __restrict__ hdr, int K, const TIn* __restrict__ x,
    const TIn* __restrict__ w, const float* __restrict__ bias, TOut* __restrict__ y, int C_in,
    int C_out, uint32_t x_bytes, Epilogue epi) {
  constexpr int NCOL = kLowCols;
  constexpr int kW = KB * kLowCin * NCOL;         // staged weights (floats)
  constexpr int kO = 4 * 64 * (NCOL + 1);         // finished rows, per wave 64 x NCOL (+1 pad)
  __shared__ float s_buf[kW > kO ? kW : kO];
  __shared__ int64_t s_row[256];
  float (*s_w)[kLowCin][NCOL] = reinterpret_cast<float (*)[kLowCin][NCOL]>(s_buf);
  const int64_t p = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  const int n0 = blockIdx.y * NCOL;               // first column of the block
  const __amdgpu_buffer_rsrc_t xr = buf_rsrc(x, x_bytes);
  const bool live = p < n_cap && p < hdr->n_out;
  const int64_t pc = p < n_cap ? p : 0;           // a position the map holds
  // the output row, loaded up front
  s_row[threadIdx.x] = live ? static_cast<int64_t>(perm[pc]) * C_out : -1;
  float acc[NCOL];
#pragma unroll
  for (int n = 0; n < NCOL; ++n) acc[n] = 0.0f;
  for (int i0 = 0; i0 < K; i0 += KB) {
    int32_t g[KB];
    load_map<KB>(gmap, gstride, K, i0, pc, g);
    float xv[KB][kLowCin];
#pragma unroll
    for (int b = 0; b < KB; ++b)
#pragma unroll
      for (int c = 0; c < kLowCin; ++c) {
        xv[b][c] = 0.0f;
        if (c < C_in && i0 + b < K) {             // block-uniform
          const uint32_t off = (live && g[b] >= 0)
                                   ? (static_cast<uint32_t>(g[b]) * C_in + c) * BufIO<TIn>::kSize
                                   : kBufOOB;
          xv[b][c] = BufIO<TIn>::load(xr, off);
        }
      }
    if (i0 > 0) __syncthreads();                  // the last batch's weights are read
    for (int e = threadIdx.x; e < KB * kLowCin * NCOL; e += blockDim.x) {
      const int b = e / (kLowCin * NCOL), c = (e / NCOL) % kLowCin, n = e % NCOL;
      s_w[b][c][n] = (i0 + b < K && c < C_in)
                         ? ElemIO<TIn>::load(w, w_index<WT>(i0 + b, K, c, n0 + n, C_in, C_out))
                         : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      if (i0 + b < K) {
        const bool has = live && g[b] >= 0;
#pragma unroll
        for (int c = 0; c < kLowCin; ++c) {
          if (c < C_in) {
#pragma unroll
            for (int n = 0; n < NCOL; ++n)
              acc[n] = has ? fmaf(xv[b][c], s_w[b][c][n], acc[n]) : acc[n];
          }
        }
      }
    }
  }
  // rows -> LDS (the weights' space), then NCOL / 4 lanes per row store
  // 4 adjacent columns each
  __syncthreads();
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  float* s_o = s_buf + wave * 64 * (NCOL + 1);
#pragma unroll
  for (int n = 0; n < NCOL; ++n) s_o[lane * (NCOL + 1) + n] = acc[n];
  __syncthreads();
  constexpr int CG = NCOL / 4;                    // 4-column groups per row
#pragma unroll
  for (int k = 0; k < CG; ++k) {
    const int idx = k * 64 + lane;
    const int r = idx / CG, cg = idx % CG;
    const int64_t o = s_row[wave * 64 + r];
    if (o < 0) continue;
    const int col = n0 + cg * 4;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = s_o[r * (NCOL + 1) + cg * 4 + e];
      if (epi.scale)
        v[e] = fmaf(v[e], epi.scale[col + e], bias ? bias[col + e] : 0.0f);
      else if (bias)
        v[e] += bias[col + e];
    }
    if (epi.res) {
      float rv[4];
      OutLoad<TOut, 4>::load(static_cast<const TOut*>(epi.res) + o + col, rv);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += rv[e];
    }
    if (epi.relu) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = v[e] < 0.0f ? 0.0f : v[e];
    }
    OutStore<TOut, 4>::store(y + o + col, v);
  }
}

// ---------------------------------------------------------------------------
// Matrix-core path
// ---------------------------------------------------------------------------
// Element traits: a lane moves 16 bytes per k-chunk; KC real k per chunk
// across the 4 lane groups of a 16x16 MFMA.
template <typename T> struct MT;
template <> struct MT<uint16_t> {          // bf16
  static constexpr int KC = 32;            // 8 bf16 per lane x 4 groups
  static constexpr int T = 8;              // transpose tile (elements per 16 B)
  __device__ static f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct MT<float> {             // fp32
  static constexpr int KC = 16;            // 4 fp32 per lane x 4 groups
  static constexpr int T = 4;
  __device__ static f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
    // The 4 elements of a lane's 16-byte chunk are consumed by 4 MFMA steps;
    // step e pairs A[r][16ch + 4g + e] with B[16ch + 4g + e][c] in every lane
    // group g, so the 4 steps cover the chunk's 16 k exactly once.
#pragma unroll
    for (int e = 0; e < 4; ++e)
      c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[e]), __uint_as_float(b[e]), c,
                                               0, 0, 0);
    return c;
  }
};

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// LDS image of W^i transposed: one row per output column of the chunk, ROWB
// bytes of k.  Rows whose length is a multiple of 128 bytes store 16-byte
// chunk c at c ^ (row & 7) (measured conflict-free for the fragment reads,
// where 16 lanes read one chunk of 16 consecutive rows; a 16-byte pad per
// row, used for other lengths, leaves a 2-way conflict).
template <int ROWB>
struct WImage {
  static constexpr bool kSwz = ROWB % 128 == 0;
  static constexpr int kRowBytes = kSwz ? ROWB : ROWB + 16;
  __device__ static int at(int row, int byte) {
    if constexpr (kSwz)
      return row * kRowBytes + ((((byte >> 4) ^ (row & 7)) << 4) | (byte & 15));
    else
      return row * kRowBytes + byte;
  }
};

// Tile of the output handled by one workgroup: 4 waves x RB blocks of 16 rows,
// NCB blocks of 16 columns (the whole workgroup shares one column chunk).
//
// Lane layout (16x16 MFMA): lane l = 16 g + r.  A operand: row r of the
// 16-row block, k-chunk bytes [16 g, 16 g + 16).  B operand: output column
// r * NCB + cb of the chunk (so a lane ends up owning NCB adjacent columns),
// same k bytes.  Result: lane l holds rows 4 g + v (v = 0..3), columns
// r * NCB + cb.
//
// Pipeline over the offsets (iteration i): G(i+3) and W^(i+2) are fetched,
// gathered rows A(i+2) are issued (their gather-map entries G(i+2) arrived
// one iteration earlier), the MFMAs of offset i run on A(i) and the LDS copy
// of W^i, and W^(i+1) (fetched one iteration earlier) is written transposed
// into the other LDS buffer.  One barrier per offset publishes W^(i+1).
template <typename TIn, int NCH, int NCB, int RB, typename TOut, int KT, bool SKIP = false,
          int WT = 0, bool LSKIP = false, bool EPI = false>
__global__ __launch_bounds__(256, 2) void k_fwd_mfma(
    const int32_t* __restrict__ gmap, const int32_t* __restrict__ perm, int64_t gstride,
    const DeviceHeader* __restrict__ hdr, int K_arg,
    const TIn* __restrict__ x, uint32_t x_bytes, const TIn* __restrict__ w,
    const float* __restrict__ bias, TOut* __restrict__ y, int C_out, int64_t ntiles,
    const int32_t* __restrict__ seg, Epilogue epi) {
  // KT > 0: the offset count is a compile-time constant and the offset loop
  // is unrolled completely (no loop-carried register hazards).
  // seg != NULL: a segmented single-offset view; this tile's weights are
  // W^seg[chunk] (tiles never straddle a chunk of kSegRows positions).
  const int K = KT > 0 ? KT : K_arg;
  constexpr int KC = MT<TIn>::KC;
  constexpr int CIN = NCH * KC;
  constexpr int COLS = NCB * 16;
  constexpr int ESZ = static_cast<int>(sizeof(TIn));
  constexpr int ROWB = CIN * ESZ;                 // bytes of one input row
  constexpr int LDWB = WImage<ROWB>::kRowBytes;   // LDS row of W^T (bytes)
  // W^T staging tasks: bf16 takes 2 k-rows x 8 columns (packed in pairs),
  // fp32 1 k-row x 4 columns; each task is one 16-byte load per k-row.
  constexpr int KPT = ESZ == 2 ? 2 : 1;           // k-rows per task
  constexpr int NPT = 16 / ESZ;                   // columns per task
  constexpr int NTASK = (CIN / KPT) * (COLS / NPT);
  constexpr int TPT = (NTASK + 255) / 256;        // tasks per thread
  constexpr int WAVE_ROWS = RB * 16;
  constexpr int TILE_ROWS = 4 * WAVE_ROWS;

  __shared__ __attribute__((aligned(16))) unsigned char s_w[2][COLS * LDWB];

  // XCD-aware tile order: workgroup b runs on XCD b % 8; give each XCD a
  // contiguous range of tiles so neighbouring tiles share that XCD's L2.  The
  // grid is sized for a bound on the rows (an SC output count is known only
  // on the device), so the ranges split the device-side tile count, not the
  // grid: otherwise a loose bound would leave whole XCDs without work.
  const int64_t n_rows = hdr->n_out;
  const int64_t nt_real = (n_rows + TILE_ROWS - 1) / TILE_ROWS;
  const int64_t nt = nt_real < ntiles ? nt_real : ntiles;
  const int64_t per = (nt + 7) / 8;
  const int64_t q = blockIdx.x / 8;
  if (q >= per) return;
  const int64_t tile = static_cast<int64_t>(blockIdx.x % 8) * per + q;
  if (tile >= nt) return;
  static_assert(kSegRows % TILE_ROWS == 0, "tiles inside one segment chunk");
  const int wseg = seg ? seg[tile * TILE_ROWS / kSegRows] : -1;

  const int col0 = blockIdx.y * COLS;
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int lr = lane % 16, lg = lane / 16;
  const int64_t row0 = tile * TILE_ROWS + wave * WAVE_ROWS;

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<TIn*>(x), 0, static_cast<int>(x_bytes),
                                        static_cast<int>(kBufDword3));
  constexpr uint32_t kOOB = 0x80000000u;   // past any x_bytes < 2^31: reads as zero

  // ---- W^i -> registers.  WT 0: task t = (k-row group kt, column group nt)
  // with nt fastest, so consecutive lanes read one k-row of the chunk end to
  // end.  WT 1/2: w holds W^T, one memory row per output column n with all k
  // contiguous; task t = (column n, 16-byte chunk kc of that row), kc fastest.
  constexpr int NGRP = COLS / NPT;                // column groups per k-row
  constexpr int CPR = ROWB / 16;                  // 16-byte chunks per W^T row
  constexpr int NTASK_T = COLS * CPR;
  constexpr int TPT_T = (NTASK_T + 255) / 256;
  constexpr int NWR = WT == 0 ? TPT * KPT : TPT_T;
  typedef u32x4 WRegs[NWR];
  auto w_load = [&](int i, WRegs& wr) {
    if (i >= K) return;
    if constexpr (WT == 0) {
#pragma unroll
      for (int q = 0; q < TPT; ++q) {
        // tasks beyond NTASK (only when NTASK is not a multiple of 256) re-read
        // task 0 and are never stored
        const int t0 = threadIdx.x + q * 256;
        const int t = (NTASK % 256 == 0 || t0 < NTASK) ? t0 : 0;
        const int kt = t / NGRP, nt = t % NGRP;
        const int iv = wseg >= 0 ? wseg : i;
        const TIn* src = w + (static_cast<int64_t>(iv) * CIN + kt * KPT) * C_out + col0 + nt * NPT;
#pragma unroll
        for (int r = 0; r < KPT; ++r)
          wr[q * KPT + r] = *reinterpret_cast<const u32x4*>(src + static_cast<int64_t>(r) * C_out);
      }
    } else {
      const int iw = wseg >= 0 ? wseg : (WT == 1 ? K - 1 - i : i);
#pragma unroll
      for (int q = 0; q < TPT_T; ++q) {
        const int t0 = threadIdx.x + q * 256;
        const int t = (NTASK_T % 256 == 0 || t0 < NTASK_T) ? t0 : 0;
        const int n = t / CPR, kc = t % CPR;
        const TIn* src = w + (static_cast<int64_t>(iw) * C_out + col0 + n) * CIN + kc * (16 / ESZ);
        wr[q] = *reinterpret_cast<const u32x4*>(src);
      }
    }
  };
  // ---- registers -> LDS, transposed: one LDS row per column n holding
  // W^i[k][n] for all k.  Column n = NCB r + cb (lane r's cb-th column) sits
  // in LDS row 16 cb + r, so the lanes that read one fragment chunk together
  // read 16 consecutive rows (spread over the banks by WImage).
  auto w_row = [](int n) { return (n % NCB) * 16 + n / NCB; };
  auto w_store = [&](int i, const WRegs& wr) {
    if (i >= K) return;
    unsigned char* dst = s_w[i & 1];
    if constexpr (WT == 0) {
#pragma unroll
      for (int q = 0; q < TPT; ++q) {
        const int t = threadIdx.x + q * 256;
        if (NTASK % 256 == 0 || t < NTASK) {
          const int kt = t / NGRP, nt = t % NGRP;
          if constexpr (ESZ == 2) {
            // pack (W[2kt][n], W[2kt+1][n]) into one 32-bit LDS word per column
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const uint32_t a = wr[q * KPT][j / 2], b = wr[q * KPT + 1][j / 2];
              const uint32_t v = (j & 1) ? ((a >> 16) | (b & 0xffff0000u))
                                         : ((a & 0xffffu) | (b << 16));
              *reinterpret_cast<uint32_t*>(&dst[WImage<ROWB>::at(w_row(nt * 8 + j), kt * 4)]) = v;
            }
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
              *reinterpret_cast<uint32_t*>(&dst[WImage<ROWB>::at(w_row(nt * 4 + j), kt * 4)]) =
                  wr[q][j];
          }
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < TPT_T; ++q) {
        const int t = threadIdx.x + q * 256;
        if (NTASK_T % 256 == 0 || t < NTASK_T) {
          const int n = t / CPR, kc = t % CPR;
          *reinterpret_cast<u32x4*>(&dst[WImage<ROWB>::at(w_row(n), kc * 16)]) = wr[q];
        }
      }
    }
  };

  // ---- gather-map entries of this wave's rows: G[i][row0 + 16 b + r]
  typedef int32_t GRegs[RB];
  // Gather-map entries (1 + input row, 0 = none) through buffer loads: an
  // offset past the map's range reads 0, so rows past the end and offsets
  // past K need no branch (a load under a divergent branch would force a
  // full wait for every load in flight).
  const uint32_t gmap_bytes = static_cast<uint32_t>(gstride * 4);
  auto g_load = [&](int i, GRegs& g) {
    const int ic = i < K ? i : 0;
    const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(gmap + static_cast<int64_t>(ic) * gstride), 0,
        static_cast<int>(gmap_bytes), static_cast<int>(kBufDword3));
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int64_t row = row0 + b * 16 + lr;
      const uint32_t off = (i < K && row < n_rows) ? static_cast<uint32_t>(row) * 4u : kOOB;
      g[b] = static_cast<int32_t>(__builtin_amdgcn_raw_buffer_load_b32(gr, off, 0, 0)) - 1;
    }
  };
  // ---- gathered rows; returns the blocks (bit b) with at least one row
  typedef u32x4 ARegs[RB][NCH];
  auto a_load = [&](const GRegs& g, ARegs& a) -> uint32_t {
    uint32_t pres = 0;
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const uint32_t base = g[b] >= 0 ? static_cast<uint32_t>(g[b]) * ROWB + lg * 16 : kOOB;
      const bool any = __ballot(g[b] >= 0) != 0;
      if (!LSKIP || any) {
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
          a[b][ch] = buf_load16(xr, base == kOOB ? kOOB : base + ch * 64);
      } else {
        // a block with no row at this offset: no loads (its products are
        // skipped as well)
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) a[b][ch] = u32x4{0u, 0u, 0u, 0u};
      }
      if (any) pres |= 1u << b;
    }
    return pres;
  };

  f32x4 acc[RB][NCB];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[b][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto mma = [&](int i, const ARegs& a, uint32_t pres) {
    const unsigned char* sw = s_w[i & 1];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      u32x4 bw[NCB];                               // W^i fragments of chunk ch
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        bw[cb] = *reinterpret_cast<const u32x4*>(
            &sw[WImage<ROWB>::at(cb * 16 + lr, ch * 64 + lg * 16)]);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        if (SKIP && !(pres & (1u << b))) continue;   // all 16 rows lack offset i
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          acc[b][cb] = MT<TIn>::mma(a[b][ch], bw[cb], acc[b][cb]);
      }
    }
  };

  // Three rotating register sets (offsets i, i+1, i+2 modulo 3).
  GRegs g0, g1, g2;
  ARegs a0, a1, a2;
  WRegs w0, w1, w2;
  uint32_t p0 = 0, p1 = 0, p2 = 0;

  // prologue: W^0 into LDS, W^1 in registers, A(0), A(1), G(2) in flight
  g_load(0, g0);
  g_load(1, g1);
  g_load(2, g2);
  w_load(0, w0);
  w_load(1, w1);
  p0 = a_load(g0, a0);
  p1 = a_load(g1, a1);
  w_store(0, w0);
  __syncthreads();

  // iteration i uses set (i mod 3): A(i) in aU, G(i+2) in gF -> A(i+2) into aF,
  // G(i+3) into gU; W^(i+1) stored from wN, W^(i+2) loaded into wF.
  auto step = [&](int i, ARegs& aU, uint32_t& pU, ARegs& aF, uint32_t& pF, GRegs& gU,
                  GRegs& gF, WRegs& wN, WRegs& wF) {
    if (i >= K) return;
    // issue order matters: the in-order load counter lets a later wait for
    // G(i+3) or W^(i+2) leave the gathered rows issued after them in flight
    g_load(i + 3, gU);
    w_load(i + 2, wF);
    pF = a_load(gF, aF);
    mma(i, aU, pU);
    w_store(i + 1, wN);
    __syncthreads();
  };
  if constexpr (KT > 0) {
#pragma unroll
    for (int i = 0; i < KT; i += 3) {
      step(i, a0, p0, a2, p2, g0, g2, w1, w2);
      step(i + 1, a1, p1, a0, p0, g1, g0, w2, w0);
      step(i + 2, a2, p2, a1, p1, g2, g1, w0, w1);
    }
  } else {
    for (int i = 0; i < K; i += 3) {
      step(i, a0, p0, a2, p2, g0, g2, w1, w2);
      step(i + 1, a1, p1, a0, p0, g1, g0, w2, w0);
      step(i + 2, a2, p2, a1, p1, g2, g1, w0, w1);
    }
  }

  // ---- epilogue: bias (EPI: scale, residual, ReLU), round once, store NCB
  // adjacent columns per lane-row
  float bv[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) bv[cb] = bias ? bias[col0 + lr * NCB + cb] : 0.0f;
  if constexpr (!EPI) {
#pragma unroll
    for (int b = 0; b < RB; ++b) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t pos = row0 + b * 16 + lg * 4 + v;   // schedule position
        const int64_t row = pos < n_rows ? perm[pos] : -1;
        if (row >= 0) {                                   // -1: padding of a segmented view
          float o[NCB];
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) o[cb] = acc[b][cb][v] + bv[cb];
          OutStore<TOut, NCB>::store(y + row * C_out + col0 + lr * NCB, o);
        }
      }
    }
  } else {
    // the block epilogue: all output rows first, then all residual loads (a
    // row of -1, padding, reads row 0, which exists whenever this tile runs),
    // so that their latencies overlap instead of one per store
    float sv[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) sv[cb] = epi.scale ? epi.scale[col0 + lr * NCB + cb] : 1.0f;
    int64_t rows[RB][4];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t pos = row0 + b * 16 + lg * 4 + v;
        rows[b][v] = pos < n_rows ? perm[pos] : -1;
      }
    const TOut* res = static_cast<const TOut*>(epi.res);
    float r[RB][4][NCB];
    if (res) {
#pragma unroll
      for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int64_t row = rows[b][v] >= 0 ? rows[b][v] : 0;
          OutLoad<TOut, NCB>::load(res + row * C_out + col0 + lr * NCB, r[b][v]);
        }
    }
#pragma unroll
    for (int b = 0; b < RB; ++b) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = rows[b][v];
        if (row >= 0) {
          float o[NCB];
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            o[cb] = epi.scale ? fmaf(acc[b][cb][v], sv[cb], bv[cb]) : acc[b][cb][v] + bv[cb];
          if (res) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) o[cb] += r[b][v][cb];
          }
          if (epi.relu) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) o[cb] = o[cb] < 0.0f ? 0.0f : o[cb];
          }
          OutStore<TOut, NCB>::store(y + row * C_out + col0 + lr * NCB, o);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------
// Row blocks per wave: fewer when the input rows are wide, so that the two
// register sets of gathered rows (current and next offset) still fit.
template <int NCH>
constexpr int rows_blocks() { return NCH <= 2 ? 4 : (NCH <= 4 ? 2 : 1); }

using Call = FwdCall;

// Tiles of fewer rows (one 16-row block per wave) when a layer is too small
// to give every compute unit two tiles of the usual size: a 64-row tile per
// workgroup keeps all of them busy on small layers (filters other than the
// unrolled 3^3 / 2^3 / 1^d ones).
constexpr int64_t kSmallLayerTiles = 512;

template <typename TIn, int NCH, int NCB, typename TOut, int WT, int RB, bool SMALL = false>
void launch_mfma_rb(const Call& c) {
  constexpr int kTileRows = 4 * RB * 16;
  const int64_t ntiles = (c.v.n_cap + kTileRows - 1) / kTileRows;
  const int64_t per = (ntiles + 7) / 8;
  dim3 grid(static_cast<unsigned>(8 * per), static_cast<unsigned>(c.C_out / (NCB * 16)));
  // Whole 16-row blocks that lack an offset skip their products.  3^3
  // filters run the unrolled kernel; other filters (strided SC, DC and the
  // SC input gradient, whose rows come ordered by offset class so that most
  // blocks take one offset only) also skip the blocks' gathers.
  // Single-offset views (f = s transposed runs, 1^d filters) unroll to one
  // step with a third of the registers, so more workgroups share a CU.
  auto kern = k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 0, true, WT, true>;
  if constexpr (!SMALL) {
    kern = c.v.K == 27  ? k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 27, true, WT>
           : c.v.K == 1 ? k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 1, true, WT>
           : c.v.K == 8 ? k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 8, true, WT, true>
                        : kern;
  }
  // The block epilogue (scale / residual / ReLU) is compiled into its own
  // kernels, so that the plain forward keeps its register count.
  if constexpr (WT == 0) {
    if (c.epi.scale || c.epi.res || c.epi.relu) {
      kern = k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 0, true, WT, true, true>;
      if constexpr (!SMALL)
        if (c.v.K == 27) kern = k_fwd_mfma<TIn, NCH, NCB, RB, TOut, 27, true, WT, false, true>;
    }
  }
  kern<<<grid, 256, 0, c.stream>>>(
      c.v.gmap, c.v.perm, c.v.gstride, c.v.hdr, static_cast<int>(c.v.K),
      static_cast<const TIn*>(c.x), c.x_bytes, static_cast<const TIn*>(c.w), c.bias,
      static_cast<TOut*>(c.y), c.C_out, ntiles, c.v.seg, c.epi);
}

template <typename TIn, int NCH, int NCB, typename TOut, int WT>
void launch_mfma(const Call& c) {
  constexpr int RB = rows_blocks<NCH>();
  const bool generic_k = c.v.K != 27 && c.v.K != 1 && c.v.K != 8;
  const int64_t tiles = (c.v.n_cap + 4 * RB * 16 - 1) / (4 * RB * 16);
  if constexpr (RB > 1) {
    if (generic_k && !c.v.seg && tiles < kSmallLayerTiles) {
      launch_mfma_rb<TIn, NCH, NCB, TOut, WT, 1, true>(c);
      return;
    }
  }
  launch_mfma_rb<TIn, NCH, NCB, TOut, WT, RB>(c);
}

template <typename TIn, int NCH, typename TOut, int WT>
void launch_mfma_ncb(const Call& c) {
  // wide fp32 rows leave no registers for 4 column blocks
  constexpr bool four = !(sizeof(TIn) == 4 && NCH >= 6);
  if (four && c.C_out % 64 == 0)
    launch_mfma<TIn, NCH, four ? 4 : 2, TOut, WT>(c);
  else if (c.C_out % 32 == 0)
    launch_mfma<TIn, NCH, 2, TOut, WT>(c);
  else
    launch_mfma<TIn, NCH, 1, TOut, WT>(c);
}

template <typename TOut, int WT>
bool try_mfma(const Call& c, int in_dt, int C_in) {
  if (c.C_out % 16 != 0) return false;
  const uint64_t xb = static_cast<uint64_t>(c.v.n_src) * C_in * (in_dt == SPCONV_BF16 ? 2 : 4);
  // buffer ranges are kept below 2^31 bytes (inputs and one offset's map row)
  if (xb >= 0x7fffffffull || static_cast<uint64_t>(c.v.gstride) * 4 >= 0x7fffffffull) return false;
  Call cc = c;
  cc.x_bytes = static_cast<uint32_t>(xb);
  if (in_dt == SPCONV_BF16) {
    switch (C_in) {
      case 32: launch_mfma_ncb<uint16_t, 1, TOut, WT>(cc); return true;
      case 64: launch_mfma_ncb<uint16_t, 2, TOut, WT>(cc); return true;
      case 96: launch_mfma_ncb<uint16_t, 3, TOut, WT>(cc); return true;
      case 128: launch_mfma_ncb<uint16_t, 4, TOut, WT>(cc); return true;
      default: return false;
    }
  }
  switch (C_in) {
    case 16: launch_mfma_ncb<float, 1, TOut, WT>(cc); return true;
    case 32: launch_mfma_ncb<float, 2, TOut, WT>(cc); return true;
    case 64: launch_mfma_ncb<float, 4, TOut, WT>(cc); return true;
    case 96: launch_mfma_ncb<float, 6, TOut, WT>(cc); return true;
    case 128: launch_mfma_ncb<float, 8, TOut, WT>(cc); return true;
    default: return false;
  }
}

template <typename TIn, typename TOut, int WT>
void launch_vec(const Call& c, int C_in) {
  const int64_t total = c.v.n_cap * c.C_out;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  k_fwd_vec<TIn, TOut, WT><<<static_cast<unsigned>(blocks), 256, 0, c.stream>>>(
      c.v.gmap, c.v.perm, c.v.gstride, c.v.n_cap, c.v.hdr, static_cast<int>(c.v.K),
      static_cast<const TIn*>(c.x), static_cast<const TIn*>(c.w), c.bias, static_cast<TOut*>(c.y),
      C_in, c.C_out, c.epi);
}

template <typename TIn, typename TOut, int WT>
void launch_lowc(const Call& c, int C_in, uint32_t x_bytes) {
  const dim3 grid(static_cast<unsigned>((c.v.n_cap + 255) / 256),
                  static_cast<unsigned>(c.C_out / kLowCols));
  // offsets in batches of KB: 9 covers a 3x3 filter in one batch (no map
  // loads for offsets past K), 16 anything larger
  auto kern = c.v.K <= 9 ? k_fwd_lowc<TIn, TOut, WT, 9> : k_fwd_lowc<TIn, TOut, WT, 16>;
  kern<<<grid, 256, 0, c.stream>>>(
      c.v.gmap, c.v.perm, c.v.gstride, c.v.n_cap, c.v.hdr, static_cast<int>(c.v.K),
      static_cast<const TIn*>(c.x), static_cast<const TIn*>(c.w), c.bias, static_cast<TOut*>(c.y),
      C_in, c.C_out, x_bytes, c.epi);
}

template <typename TIn, typename TOut, int WT>
void launch_generic(const Call& c, int C_in) {
  // one grid row of blocks per kLowCols columns (at most 65535), the inputs
  // and one offset's map row addressable by a buffer resource (< 2^31 bytes).
  // Below kLowMinRows positions the one-lane-per-column kernel finishes
  // first (measured: 460 rows of 16 columns 6.1 us against 7.7 us; 29759
  // rows of 32 columns 16.4 us against 12.7 us).
  constexpr int64_t kLowMinRows = 2048;
  const uint64_t xb = static_cast<uint64_t>(c.v.n_src) * C_in * sizeof(TIn);
  if (C_in <= kLowCin && c.v.n_cap >= kLowMinRows && c.C_out % kLowCols == 0 &&
      c.C_out / kLowCols <= 65535 &&
      xb < kBufOOB && static_cast<uint64_t>(c.v.gstride) * 4 < kBufOOB)
    launch_lowc<TIn, TOut, WT>(c, C_in, static_cast<uint32_t>(xb));
  else
    launch_vec<TIn, TOut, WT>(c, C_in);
}

template <int WT>
bool run(const Call& c, int in_dt, int out_dt, int C_in) {
  bool done = false;
  if (!force_vector_path()) {
    done = out_dt == SPCONV_F32 ? try_mfma<float, WT>(c, in_dt, C_in)
                                : try_mfma<uint16_t, WT>(c, in_dt, C_in);
  }
  if (done) return true;
  if (c.v.seg) return false;               // segmented views run on the matrix cores only
  if (in_dt == SPCONV_F32 && out_dt == SPCONV_F32)
    launch_generic<float, float, WT>(c, C_in);
  else if (in_dt == SPCONV_F32)
    launch_generic<float, uint16_t, WT>(c, C_in);
  else if (out_dt == SPCONV_F32)
    launch_generic<uint16_t, float, WT>(c, C_in);
  else
    launch_generic<uint16_t, uint16_t, WT>(c, C_in);
  return true;
}

}  // namespace
}  // namespace spc
