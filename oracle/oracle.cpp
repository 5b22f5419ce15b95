// Oracle for sparse convolution (SC) and valid sparse convolution (VSC).
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
// CPU statement of what the GPU path computes.  Only the test suite, the
// smoke check and the benchmark's CPU-baseline leg load it.  It shares no
// code, header, table or helper with the HIP library, and neither side
// includes or links the other.
//
// What it follows (Graham & van der Maaten, "Submanifold Sparse
// Convolutional Networks"):
//   * state of a layer: a map (location -> row) and a feature matrix with one
//     row per active site (Section 4, Implementation);
//   * SC(m,n,f,s): an output site is active when any input site in its f^d
//     receptive field is active; the output extent is (l - f + s)/s; the
//     ground state is replaced by zero (Section 3);
//   * VSC(m,n,f,1): input padded by (f-1)/2, output active iff the central
//     input site is active, features computed as for SC (Section 3);
//   * rule book R = (R_i), R_i a list of (input row, output row) pairs per
//     filter offset i (Section 4);
//   * forward: output matrix starts at zero; for every pair of R_i add the
//     input row times W^i to the output row (Section 4);
//   * max-pooling MP(f,s) and average-pooling AP(f,s) are variants of
//     SC(.,.,f,s): MP takes the maximum of the zero vector and the input
//     vectors of the receptive field, AP f^-d times the sum of the active
//     input vectors (Section 3);
//   * deconvolution DC(.,.,f,s) inverts SC(.,.,f,s): its active output sites
//     are the SC input sites and every connection is reversed (Section 3);
//   * the backward pass (the networks of Section 5 are trained with SGD) is
//     the derivative of the forward sums: input gradients run every pair in
//     the opposite direction with W^i transposed, weight gradients sum
//     input-row x output-gradient-row outer products over R_i.
//
// Readings where the paper is silent (each one is listed in the design notes):
//   * coordinate 0 is the sample index, with f[0] = s[0] = 1, so samples never
//     interact;
//   * SC takes any f >= 1, s >= 1 with no padding: extent floor((l-f)/s)+1;
//   * W^i multiplies the input at s*y + i (SC) or y + i - (f-1)/2 (VSC): a
//     cross-correlation, offsets flattened row-major (last dimension fastest);
//   * SC output rows are numbered in lexicographic order of the output site;
//   * pairs inside R_i are ordered by ascending output row (each output row
//     has at most one input per offset, so this is a total order);
//   * the bias (optional) is added once at every active output site;
//   * accumulation is in double, rounded once to the output type (RNE);
//   * MP and AP run on an SC rule book; f^-d is 1 / prod_j f_j over the
//     spatial dimensions (non-square filters); MP compares with IEEE maxNum
//     (a NaN input is ignored), so its result is never NaN;
//   * DC runs on an SC rule book (DC is defined as the inverse of SC).
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <vector>

#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

enum { OK = 0, EINVAL_ = -1, EDUP_ = -2, ERANGE_ = -3 };
enum { VSC = 0, SC = 1, DC = 2 };
enum { POOL_MAX = 0, POOL_AVG = 1 };
enum { F32 = 0, BF16 = 1 };

using Site = std::array<int32_t, 4>;   // unused trailing entries are 0

struct Rulebook {
  int kind = 0, D = 0;
  int64_t n_in = 0, n_out = 0, K = 0;
  std::vector<int32_t> f, s, in_size, out_size;
  std::vector<int32_t> out_coords;                       // [n_out][D]
  std::vector<std::vector<std::array<int64_t, 2>>> R;    // R[i] = (in, out)
};

double bf16_to_double(uint16_t b) {
  uint32_t u = static_cast<uint32_t>(b) << 16;
  float v;
  std::memcpy(&v, &u, 4);
  return static_cast<double>(v);
}

double load(int dt, const void* p, int64_t idx) {
  if (dt == F32) return static_cast<double>(static_cast<const float*>(p)[idx]);
  return bf16_to_double(static_cast<const uint16_t*>(p)[idx]);
}

// Offset index i (flattened, last dimension fastest) -> per-dimension offset.
void unflatten(int64_t i, int D, const std::vector<int32_t>& f, int32_t* o) {
  for (int j = D - 1; j >= 0; --j) {
    o[j] = static_cast<int32_t>(i % f[j]);
    i /= f[j];
  }
}

}  // namespace

extern "C" {

// Build the rule book of a VSC (kind 0) or SC (kind 1) layer.
//   coords  host int32 [N][D], coordinate 0 = sample index
//   size    host int32 [D], grid extent per dimension (size[0] = sample count)
//   f, s    host int32 [D], filter size and stride, f[0] = s[0] = 1
// Returns 0 and a handle in *out, or a negative status (EINVAL -1, EDUP -2,
// ERANGE -3) with *out = NULL.
int ref_build(int kind, int D, const int32_t* coords, int64_t N,
              const int32_t* size, const int32_t* f, const int32_t* s,
              void** out) {
  *out = nullptr;
  if (kind != VSC && kind != SC) return EINVAL_;
  if (D < 2 || D > 4 || N < 0 || (N > 0 && !coords)) return EINVAL_;
  if (!size || !f || !s) return EINVAL_;
  if (f[0] != 1 || s[0] != 1) return EINVAL_;
  for (int j = 0; j < D; ++j) {
    if (size[j] < 1 || size[j] > 65535 || f[j] < 1 || s[j] < 1) return EINVAL_;
    if (kind == VSC && (f[j] % 2 != 1 || s[j] != 1)) return EINVAL_;
  }

  auto* rb = new Rulebook;
  rb->kind = kind;
  rb->D = D;
  rb->n_in = N;
  rb->f.assign(f, f + D);
  rb->s.assign(s, s + D);
  rb->in_size.assign(size, size + D);
  rb->K = 1;
  for (int j = 0; j < D; ++j) rb->K *= f[j];

  // Range check of every row first, then the input map (location -> row);
  // a location given twice is an error, never merged.
  for (int64_t r = 0; r < N; ++r)
    for (int j = 0; j < D; ++j)
      if (coords[r * D + j] < 0 || coords[r * D + j] >= size[j]) {
        delete rb;
        return ERANGE_;
      }
  std::map<Site, int64_t> in_map;
  for (int64_t r = 0; r < N; ++r) {
    Site x{0, 0, 0, 0};
    for (int j = 0; j < D; ++j) x[j] = coords[r * D + j];
    if (!in_map.emplace(x, r).second) {
      delete rb;
      return EDUP_;
    }
  }

  // Output sites, in output-row order.
  std::vector<Site> out_sites;
  if (kind == VSC) {
    rb->out_size = rb->in_size;
    out_sites.resize(N);
    for (int64_t r = 0; r < N; ++r) {
      Site x{0, 0, 0, 0};
      for (int j = 0; j < D; ++j) x[j] = coords[r * D + j];
      out_sites[r] = x;        // output row r is input row r
    }
  } else {
    rb->out_size.resize(D);
    for (int j = 0; j < D; ++j)
      rb->out_size[j] = size[j] >= f[j] ? (size[j] - f[j]) / s[j] + 1 : 0;
    // y is active when some active input x = s*y + i with 0 <= i < f exists,
    // i.e. t = x - i is a non-negative multiple of s inside the output grid.
    std::set<Site> ys;
    std::vector<int32_t> o(D);
    for (const auto& kv : in_map) {
      for (int64_t i = 0; i < rb->K; ++i) {
        unflatten(i, D, rb->f, o.data());
        Site y{0, 0, 0, 0};
        bool ok = true;
        for (int j = 0; j < D && ok; ++j) {
          int32_t t = kv.first[j] - o[j];
          if (t < 0 || t % s[j] != 0 || t / s[j] >= rb->out_size[j]) ok = false;
          else y[j] = t / s[j];
        }
        if (ok) ys.insert(y);
      }
    }
    out_sites.assign(ys.begin(), ys.end());   // lexicographic order
  }
  rb->n_out = static_cast<int64_t>(out_sites.size());
  rb->out_coords.resize(rb->n_out * D);
  for (int64_t r = 0; r < rb->n_out; ++r)
    for (int j = 0; j < D; ++j) rb->out_coords[r * D + j] = out_sites[r][j];

  // Rule book: for every offset i and every output row y, in ascending order,
  // the input site feeding y through W^i, if active.  The lookups of one
  // offset are independent read-only map queries (run in parallel over y);
  // the list is then appended in row order, so R_i does not depend on the
  // thread count.
  rb->R.resize(rb->K);
  std::vector<int64_t> found(rb->n_out);
  for (int64_t i = 0; i < rb->K; ++i) {
    int32_t o[4] = {0, 0, 0, 0};
    unflatten(i, D, rb->f, o);
#pragma omp parallel for schedule(static)
    for (int64_t y = 0; y < rb->n_out; ++y) {
      Site x{0, 0, 0, 0};
      for (int j = 0; j < D; ++j) {
        if (kind == VSC) x[j] = out_sites[y][j] + o[j] - (f[j] - 1) / 2;
        else x[j] = s[j] * out_sites[y][j] + o[j];
      }
      auto it = in_map.find(x);
      found[y] = it == in_map.end() ? -1 : it->second;
    }
    for (int64_t y = 0; y < rb->n_out; ++y)
      if (found[y] >= 0) rb->R[i].push_back({found[y], y});
  }
  *out = rb;
  return OK;
}

// Sizes of a built rule book.  out_size: host int32 [D] or NULL;
// pair_off: host int64 [K+1] (prefix sums of k_i) or NULL.
int ref_query(void* h, int64_t* n_in, int64_t* n_out, int64_t* K,
              int32_t* out_size, int64_t* pair_off) {
  if (!h) return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (n_in) *n_in = rb->n_in;
  if (n_out) *n_out = rb->n_out;
  if (K) *K = rb->K;
  if (out_size)
    for (int j = 0; j < rb->D; ++j) out_size[j] = rb->out_size[j];
  if (pair_off) {
    pair_off[0] = 0;
    for (int64_t i = 0; i < rb->K; ++i)
      pair_off[i + 1] = pair_off[i] + static_cast<int64_t>(rb->R[i].size());
  }
  return OK;
}

// Output coordinates (host int32 [n_out][D]) and pairs (host int32 [sum k][2],
// R_0 first, each R_i in Z-order of the output site).  Either may be NULL.
int ref_export(void* h, int32_t* out_coords, int32_t* pairs) {
  if (!h) return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (out_coords)
    for (size_t k = 0; k < rb->out_coords.size(); ++k)
      out_coords[k] = rb->out_coords[k];
  if (pairs) {
    int64_t p = 0;
    for (const auto& Ri : rb->R)
      for (const auto& pr : Ri) {
        pairs[2 * p] = static_cast<int32_t>(pr[0]);
        pairs[2 * p + 1] = static_cast<int32_t>(pr[1]);
        ++p;
      }
  }
  return OK;
}

}  // extern "C"

namespace {

// For every offset i and output row y, the input row R_i pairs with y, or -1
// (each output row has at most one input per offset).
std::vector<int64_t> source_rows(const Rulebook& rb) {
  std::vector<int64_t> src(static_cast<size_t>(rb.K * rb.n_out), -1);
  for (int64_t i = 0; i < rb.K; ++i)
    for (const auto& pr : rb.R[i]) src[i * rb.n_out + pr[1]] = pr[0];
  return src;
}

// The forward multiply-add of Section 4 for one output row yo: start from the
// bias, then add input row times W^i for every offset i in ascending order,
// input plane c in ascending order, all in double.
void forward_row(int64_t yo, const int64_t* src, int64_t K, int64_t n_out, int in_dt,
                 const void* x, const void* w, const float* bias, int C_in, int C_out,
                 double* y, double* absb, const double* x_absb) {
  double* yr = y + yo * C_out;
  double* ar = absb ? absb + yo * C_out : nullptr;
  for (int n = 0; n < C_out; ++n) {
    const double b = bias ? static_cast<double>(bias[n]) : 0.0;
    yr[n] = b;
    if (ar) ar[n] = std::fabs(b);
  }
  for (int64_t i = 0; i < K; ++i) {
    const int64_t xi = src[i * n_out + yo];
    if (xi < 0) continue;
    for (int c = 0; c < C_in; ++c) {
      const double xv = load(in_dt, x, xi * C_in + c);
      const double xa = x_absb ? x_absb[xi * C_in + c] : std::fabs(xv);
      for (int n = 0; n < C_out; ++n) {
        const double wv = load(in_dt, w, (i * C_in + c) * C_out + n);
        yr[n] += xv * wv;
        if (ar) ar[n] += xa * std::fabs(wv);
      }
    }
  }
}

// The forward for the output rows with rows_mask[y] != 0 (every row when
// rows_mask is NULL).  Rows are independent and each row's sum has one fixed
// order, so the result does not depend on how many threads share the rows.
void forward_impl(const Rulebook& rb, int in_dt, const void* x, const void* w,
                  const float* bias, int C_in, int C_out, const uint8_t* rows_mask,
                  double* y, double* absb, const double* x_absb) {
  const std::vector<int64_t> src = source_rows(rb);
  const int64_t K = rb.K, n_out = rb.n_out;
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t yo = 0; yo < n_out; ++yo) {
    if (rows_mask && !rows_mask[yo]) continue;
    forward_row(yo, src.data(), K, n_out, in_dt, x, w, bias, C_in, C_out, y, absb, x_absb);
  }
}

}  // namespace

extern "C" {

// Forward pass.  x: host [n_in][C_in] of in_dt (0 = fp32, 1 = bf16 bits);
// w: host [K][C_in][C_out] of in_dt; bias: host fp32 [C_out] or NULL.
// y: host double [n_out][C_out], the exact-as-double result.
// absb: host double [n_out][C_out] or NULL: |bias| + sum |x||w|, the scale the
// tolerance is measured against.  x_absb: host double [n_in][C_in] or NULL; if
// given it replaces |x| in absb (bounds carried through a stack of layers).
int ref_forward(void* h, int in_dt, const void* x, const void* w,
                const float* bias, int C_in, int C_out, double* y,
                double* absb, const double* x_absb) {
  if (!h || C_in < 1 || C_out < 1 || (in_dt != F32 && in_dt != BF16))
    return EINVAL_;
  forward_impl(*static_cast<Rulebook*>(h), in_dt, x, w, bias, C_in, C_out, nullptr, y, absb,
               x_absb);
  return OK;
}

// Same as ref_forward restricted to the output rows with rows_mask[y] != 0
// (host uint8 [n_out]); other rows of y / absb are left untouched.  Lets a
// test check sampled rows of a layer too large for the full CPU forward.
int ref_forward_rows(void* h, int in_dt, const void* x, const void* w,
                     const float* bias, int C_in, int C_out,
                     const uint8_t* rows_mask, double* y, double* absb) {
  if (!h || !rows_mask || !absb || C_in < 1 || C_out < 1 ||
      (in_dt != F32 && in_dt != BF16))
    return EINVAL_;
  forward_impl(*static_cast<Rulebook*>(h), in_dt, x, w, bias, C_in, C_out, rows_mask, y, absb,
               nullptr);
  return OK;
}

// Threads the parallel loops above may use (0 or less: the OpenMP default).
// Returns the count now in effect (1 when built without OpenMP).
int ref_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

// Sparse pooling on an SC rule book.
//   mode   POOL_MAX (MP) or POOL_AVG (AP)
//   x      host [n_in][C] of dt (fp32 or bf16 bits)
//   y      host double [n_out][C]; absb host double [n_out][C] or NULL (AP:
//          sum |x| / K, the tolerance scale; MP: |y|)
int ref_pool(void* h, int mode, int dt, const void* x, int C, double* y, double* absb) {
  if (!h || C < 1 || (dt != F32 && dt != BF16) || (mode != POOL_MAX && mode != POOL_AVG))
    return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (rb->kind != SC) return EINVAL_;
  for (int64_t r = 0; r < rb->n_out * C; ++r) {
    y[r] = 0.0;                        // MP: the zero vector; AP: empty sum
    if (absb) absb[r] = 0.0;
  }
  for (int64_t i = 0; i < rb->K; ++i)
    for (const auto& pr : rb->R[i])
      for (int c = 0; c < C; ++c) {
        const double v = load(dt, x, pr[0] * C + c);
        double& o = y[pr[1] * C + c];
        if (mode == POOL_MAX) {
          o = std::fmax(o, v);
        } else {
          o += v;
          if (absb) absb[pr[1] * C + c] += std::fabs(v);
        }
      }
  if (mode == POOL_AVG) {
    const double k = static_cast<double>(rb->K);   // prod_j f_j, f_0 = 1
    for (int64_t r = 0; r < rb->n_out * C; ++r) {
      y[r] /= k;
      if (absb) absb[r] /= k;
    }
  } else if (absb) {
    for (int64_t r = 0; r < rb->n_out * C; ++r) absb[r] = std::fabs(y[r]);
  }
  return OK;
}

// DC forward on an SC rule book: output rows are the SC input rows.
//   x     host [n_out][C_in] of dt (features on the SC output sites)
//   w     host [K][C_in][C_out] of dt; bias host fp32 [C_out] or NULL
//   y     host double [n_in][C_out]: bias + sum_i sum_{(a,b) in R_i} x[b] W^i
//         into row a;  absb / x_absb as for ref_forward
int ref_dc_forward(void* h, int dt, const void* x, const void* w, const float* bias,
                   int C_in, int C_out, double* y, double* absb, const double* x_absb) {
  if (!h || C_in < 1 || C_out < 1 || (dt != F32 && dt != BF16)) return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (rb->kind != SC) return EINVAL_;
  for (int64_t r = 0; r < rb->n_in; ++r)
    for (int n = 0; n < C_out; ++n) {
      const double b = bias ? static_cast<double>(bias[n]) : 0.0;
      y[r * C_out + n] = b;
      if (absb) absb[r * C_out + n] = std::fabs(b);
    }
  for (int64_t i = 0; i < rb->K; ++i)
    for (const auto& pr : rb->R[i]) {
      const int64_t src = pr[1], dst = pr[0];       // the SC pair read backwards
      for (int c = 0; c < C_in; ++c) {
        const double xv = load(dt, x, src * C_in + c);
        const double xa = x_absb ? x_absb[src * C_in + c] : std::fabs(xv);
        for (int n = 0; n < C_out; ++n) {
          const double wv = load(dt, w, (i * C_in + c) * C_out + n);
          y[dst * C_out + n] += xv * wv;
          if (absb) absb[dst * C_out + n] += xa * std::fabs(wv);
        }
      }
    }
  return OK;
}

// Gradient with respect to the layer input, given the gradient dy of its
// output and the weights w [K][C_in][C_out] (dt).
//   op VSC / SC (rule book of that kind): dx [n_in][C_in],
//      dx[a] = sum_i sum_{(a,b) in R_i} dy[b] (W^i)^T, dy [n_out][C_out]
//   op DC (SC rule book): dx [n_out][C_in],
//      dx[b] = sum_i sum_{(a,b) in R_i} dy[a] (W^i)^T, dy [n_in][C_out]
//   dx, absb: host double; absb = sum |dy| |w| (the tolerance scale) or NULL
int ref_backward_data(void* h, int op, int dt, const void* dy, const void* w, int C_in,
                      int C_out, double* dx, double* absb) {
  if (!h || C_in < 1 || C_out < 1 || (dt != F32 && dt != BF16)) return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (op == DC ? rb->kind != SC : op != rb->kind) return EINVAL_;
  const int64_t rows = op == DC ? rb->n_out : rb->n_in;
  for (int64_t r = 0; r < rows * C_in; ++r) {
    dx[r] = 0.0;
    if (absb) absb[r] = 0.0;
  }
  for (int64_t i = 0; i < rb->K; ++i)
    for (const auto& pr : rb->R[i]) {
      const int64_t src = op == DC ? pr[0] : pr[1];   // row of dy
      const int64_t dst = op == DC ? pr[1] : pr[0];   // row of dx
      for (int n = 0; n < C_out; ++n) {
        const double g = load(dt, dy, src * C_out + n);
        for (int c = 0; c < C_in; ++c) {
          const double wv = load(dt, w, (i * C_in + c) * C_out + n);
          dx[dst * C_in + c] += g * wv;
          if (absb) absb[dst * C_in + c] += std::fabs(g) * std::fabs(wv);
        }
      }
    }
  return OK;
}

// Gradients of the weights and the bias, given the layer input x and the
// output gradient dy (both dt).
//   op VSC / SC: x [n_in][C_in], dy [n_out][C_out],
//      dw[i][c][n] = sum_{(a,b) in R_i} x[a][c] dy[b][n]
//   op DC (SC rule book): x [n_out][C_in], dy [n_in][C_out],
//      dw[i][c][n] = sum_{(a,b) in R_i} x[b][c] dy[a][n]
//   db[n] = sum of dy[.][n] over all output rows (NULL: skipped)
//   dw / db / absb_w / absb_b: host double; absb_* (sum of |terms|) or NULL
//   omask: host [K], nonzero = compute dw for that offset (others stay 0);
//          NULL = every offset
int ref_backward_weight(void* h, int op, int dt, const void* x, const void* dy, int C_in,
                        int C_out, double* dw, double* db, double* absb_w, double* absb_b,
                        const uint8_t* omask) {
  if (!h || C_in < 1 || C_out < 1 || (dt != F32 && dt != BF16)) return EINVAL_;
  auto* rb = static_cast<Rulebook*>(h);
  if (op == DC ? rb->kind != SC : op != rb->kind) return EINVAL_;
  const int64_t nw = rb->K * C_in * C_out;
  for (int64_t k = 0; k < nw; ++k) {
    dw[k] = 0.0;
    if (absb_w) absb_w[k] = 0.0;
  }
  // Every entry (i, c, n) sums over the pairs of R_i in list order; the
  // entries of different (i, c) are independent and run in parallel, so the
  // result does not depend on the thread count.
  const int64_t K = rb->K;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int64_t i = 0; i < K; ++i)
    for (int c = 0; c < C_in; ++c) {
      if (omask && !omask[i]) continue;
      double* dwr = dw + (i * C_in + c) * C_out;
      double* awr = absb_w ? absb_w + (i * C_in + c) * C_out : nullptr;
      for (const auto& pr : rb->R[i]) {
        const int64_t xr = op == DC ? pr[1] : pr[0];
        const int64_t gr = op == DC ? pr[0] : pr[1];
        const double xv = load(dt, x, xr * C_in + c);
        for (int n = 0; n < C_out; ++n) {
          const double g = load(dt, dy, gr * C_out + n);
          dwr[n] += xv * g;
          if (awr) awr[n] += std::fabs(xv) * std::fabs(g);
        }
      }
    }
  if (db) {
    const int64_t out_rows = op == DC ? rb->n_in : rb->n_out;
    for (int n = 0; n < C_out; ++n) {
      double s = 0.0, a = 0.0;
      for (int64_t r = 0; r < out_rows; ++r) {
        const double g = load(dt, dy, r * C_out + n);
        s += g;
        a += std::fabs(g);
      }
      db[n] = s;
      if (absb_b) absb_b[n] = a;
    }
  }
  return OK;
}

// Round doubles once to the output type: fp32 (out: float*) or bf16 (out:
// uint16_t* bit patterns), both round-to-nearest-even.
int ref_round(const double* v, int64_t n, int out_dt, void* out) {
  if (out_dt == F32) {
    for (int64_t k = 0; k < n; ++k)
      static_cast<float*>(out)[k] = static_cast<float>(v[k]);
    return OK;
  }
  if (out_dt != BF16) return EINVAL_;
  for (int64_t k = 0; k < n; ++k) {
    double d = v[k];
    float r;
    if (std::isnan(d)) {
      r = std::nanf("");
    } else if (d == 0.0 || std::isinf(d)) {
      r = static_cast<float>(d);
    } else {
      // bf16 keeps 8 significant bits; below 2^-126 the quantum is 2^-133.
      int e;
      std::frexp(d, &e);                       // |d| = m 2^e, 0.5 <= m < 1
      int qe = e - 8 < -133 ? -133 : e - 8;
      double q = std::nearbyint(std::ldexp(d, -qe));   // ties to even
      double rd = std::ldexp(q, qe);
      const double bf16_max = 3.3895313892515355e38;  // (2^8 - 1) 2^120
      if (std::fabs(rd) > bf16_max) rd = std::copysign(INFINITY, d);
      r = static_cast<float>(rd);              // exact: rd is a bf16 value
    }
    uint32_t u;
    std::memcpy(&u, &r, 4);
    static_cast<uint16_t*>(out)[k] = static_cast<uint16_t>(u >> 16);
  }
  return OK;
}

void ref_free(void* h) { delete static_cast<Rulebook*>(h); }

}  // extern "C"
