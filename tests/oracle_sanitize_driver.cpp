// Exercises every oracle entry point on small random layers, for a build with
// AddressSanitizer and UndefinedBehaviorSanitizer (host code only; see
// tests/test_oracle_sanitized.py).  Exit code 0 when every call returned the
// status it should; the sanitizers abort on a memory or UB error.
#include <cstdint>
#include <cstdio>
#include <random>
#include <set>
#include <vector>

extern "C" {
int ref_build(int kind, int D, const int32_t* coords, int64_t N, const int32_t* size,
              const int32_t* f, const int32_t* s, void** out);
int ref_query(void* h, int64_t* n_in, int64_t* n_out, int64_t* K, int32_t* out_size,
              int64_t* pair_off);
int ref_export(void* h, int32_t* out_coords, int32_t* pairs);
int ref_forward(void* h, int in_dt, const void* x, const void* w, const float* bias, int C_in,
                int C_out, double* y, double* absb, const double* x_absb);
int ref_forward_rows(void* h, int in_dt, const void* x, const void* w, const float* bias,
                     int C_in, int C_out, const uint8_t* rows_mask, double* y, double* absb);
int ref_pool(void* h, int mode, int dt, const void* x, int C, double* y, double* absb);
int ref_dc_forward(void* h, int dt, const void* x, const void* w, const float* bias, int C_in,
                   int C_out, double* y, double* absb, const double* x_absb);
int ref_backward_data(void* h, int op, int dt, const void* dy, const void* w, int C_in,
                      int C_out, double* dx, double* absb);
int ref_backward_weight(void* h, int op, int dt, const void* x, const void* dy, int C_in,
                        int C_out, double* dw, double* db, double* absb_w, double* absb_b,
                        const uint8_t* omask);
int ref_round(const double* v, int64_t n, int out_dt, void* out);
void ref_free(void* h);
}

static int failures = 0;
static void expect(bool ok, const char* what) {
  if (!ok) {
    std::printf("FAILED: %s\n", what);
    ++failures;
  }
}

static std::vector<int32_t> sites(std::mt19937& g, int D, const int32_t* size, double density) {
  std::vector<int32_t> c;
  std::vector<int32_t> x(D, 0);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  while (true) {
    if (u(g) < density) c.insert(c.end(), x.begin(), x.end());
    int j = D - 1;
    while (j >= 0 && ++x[j] == size[j]) x[j--] = 0;
    if (j < 0) break;
  }
  return c;
}

static void layer(std::mt19937& g, int kind, int D, const int32_t* size, const int32_t* f,
                  const int32_t* s, double density) {
  std::vector<int32_t> c = sites(g, D, size, density);
  const int64_t N = static_cast<int64_t>(c.size()) / D;
  void* h = nullptr;
  expect(ref_build(kind, D, c.data(), N, size, f, s, &h) == 0 && h, "build");
  int64_t n_in = 0, n_out = 0, K = 0;
  std::vector<int32_t> osz(D);
  expect(ref_query(h, &n_in, &n_out, &K, osz.data(), nullptr) == 0, "query");
  std::vector<int64_t> off(K + 1);
  ref_query(h, nullptr, nullptr, nullptr, nullptr, off.data());
  std::vector<int32_t> oc(static_cast<size_t>(n_out * D) + 1), pairs(2 * off[K] + 2);
  expect(ref_export(h, oc.data(), pairs.data()) == 0, "export");
  const int Ci = 3, Co = 2;
  std::normal_distribution<float> nd;
  std::vector<float> x(n_in * Ci + 1), w(K * Ci * Co), b(Co), dy(n_out * Co + 1);
  for (auto& v : x) v = nd(g);
  for (auto& v : w) v = nd(g);
  for (auto& v : b) v = nd(g);
  for (auto& v : dy) v = nd(g);
  std::vector<uint16_t> xb(x.size());
  for (size_t i = 0; i < x.size(); ++i) xb[i] = static_cast<uint16_t>(
      *reinterpret_cast<const uint32_t*>(&x[i]) >> 16);
  std::vector<uint16_t> wb(w.size());
  for (size_t i = 0; i < w.size(); ++i) wb[i] = static_cast<uint16_t>(
      *reinterpret_cast<const uint32_t*>(&w[i]) >> 16);
  std::vector<double> y(n_out * Co + 1), a(n_out * Co + 1);
  expect(ref_forward(h, 0, x.data(), w.data(), b.data(), Ci, Co, y.data(), a.data(), nullptr) == 0,
         "forward f32");
  expect(ref_forward(h, 1, xb.data(), wb.data(), nullptr, Ci, Co, y.data(), a.data(), nullptr) ==
             0, "forward bf16");
  std::vector<uint8_t> mask(n_out + 1, 1);
  expect(ref_forward_rows(h, 0, x.data(), w.data(), b.data(), Ci, Co, mask.data(), y.data(),
                          a.data()) == 0, "forward rows");
  std::vector<float> yr(n_out * Co + 1);
  std::vector<uint16_t> yb(n_out * Co + 1);
  expect(ref_round(y.data(), n_out * Co, 0, yr.data()) == 0, "round f32");
  expect(ref_round(y.data(), n_out * Co, 1, yb.data()) == 0, "round bf16");
  std::vector<double> dx(n_in * Ci + 1), ax(n_in * Ci + 1);
  expect(ref_backward_data(h, kind, 0, dy.data(), w.data(), Ci, Co, dx.data(), ax.data()) == 0,
         "backward data");
  std::vector<double> dw(K * Ci * Co), db(Co), aw(K * Ci * Co), ab(Co);
  expect(ref_backward_weight(h, kind, 0, x.data(), dy.data(), Ci, Co, dw.data(), db.data(),
                             aw.data(), ab.data(), nullptr) == 0, "backward weight");
  if (kind == 1) {
    std::vector<double> py(n_out * Ci + 1), pa(n_out * Ci + 1);
    expect(ref_pool(h, 0, 0, x.data(), Ci, py.data(), pa.data()) == 0, "max pool");
    expect(ref_pool(h, 1, 1, xb.data(), Ci, py.data(), pa.data()) == 0, "avg pool");
    // DC: inputs on the SC output sites, outputs on the SC input sites
    std::vector<float> xd(n_out * Ci + 1);
    for (auto& v : xd) v = nd(g);
    std::vector<double> yd(n_in * Co + 1), ad(n_in * Co + 1);
    expect(ref_dc_forward(h, 0, xd.data(), w.data(), b.data(), Ci, Co, yd.data(), ad.data(),
                          nullptr) == 0, "dc forward");
    std::vector<float> dyd(n_in * Co + 1);
    for (auto& v : dyd) v = nd(g);
    std::vector<double> dxd(n_out * Ci + 1), axd(n_out * Ci + 1);
    expect(ref_backward_data(h, 2, 0, dyd.data(), w.data(), Ci, Co, dxd.data(), axd.data()) == 0,
           "dc backward data");
    expect(ref_backward_weight(h, 2, 0, xd.data(), dyd.data(), Ci, Co, dw.data(), db.data(),
                               nullptr, nullptr, nullptr) == 0, "dc backward weight");
  } else {
    expect(ref_pool(h, 0, 0, x.data(), Ci, y.data(), a.data()) != 0, "pool on a VSC book");
  }
  ref_free(h);
}

int main() {
  std::mt19937 g(7);
  for (int rep = 0; rep < 3; ++rep) {
    const int32_t s2[3] = {2, 9, 7}, f3[3] = {1, 3, 3}, one[3] = {1, 1, 1};
    layer(g, 0, 3, s2, f3, one, 0.3);
    const int32_t s3[4] = {2, 6, 5, 7}, f5[4] = {1, 5, 3, 1}, ones[4] = {1, 1, 1, 1};
    layer(g, 0, 4, s3, f5, ones, 0.2);
    const int32_t fs[4] = {1, 2, 2, 2}, ss[4] = {1, 2, 2, 2};
    layer(g, 1, 4, s3, fs, ss, 0.4);
    const int32_t fo[3] = {1, 3, 2}, so[3] = {1, 2, 3};
    layer(g, 1, 3, s2, fo, so, 0.5);
    layer(g, 1, 3, s2, fo, so, 0.0);                 // no sites
  }
  // errors: duplicate site, out of range, even VSC filter
  const int32_t size[3] = {1, 4, 4}, f[3] = {1, 3, 3}, s[3] = {1, 1, 1}, fe[3] = {1, 2, 2};
  const int32_t dup[6] = {0, 1, 1, 0, 1, 1}, oor[3] = {0, 4, 0}, ok[3] = {0, 1, 1};
  void* h = nullptr;
  expect(ref_build(0, 3, dup, 2, size, f, s, &h) == -2 && !h, "duplicate");
  expect(ref_build(0, 3, oor, 1, size, f, s, &h) == -3 && !h, "out of range");
  expect(ref_build(0, 3, ok, 1, size, fe, s, &h) == -1 && !h, "even filter");
  std::printf("%s\n", failures ? "errors" : "ok");
  return failures ? 1 : 0;
}
