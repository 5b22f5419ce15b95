// C ABI of the sparse-convolution library: argument validation, rule-book
// lifetime and memory, synchronisation, and dispatch to the HIP kernels.
// Every entry point returns a status code; nothing is printed.
#include <cstring>
#include <mutex>
#include <new>

#include "internal.h"

namespace spc {

Codec make_codec(int D, const int32_t* size) {
  Codec c{};
  c.D = D;
  int sh = 0;
  for (int j = D - 1; j >= 0; --j) {
    const int b = bitlen(static_cast<uint64_t>(size[j] > 0 ? size[j] - 1 : 0));
    c.shift[j] = sh;
    c.fmask[j] = b ? ((1u << b) - 1u) : 0u;
    c.size[j] = size[j];
    sh += b;
  }
  c.kbits = sh;
  return c;
}

}  // namespace spc

namespace {

using namespace spc;

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int status_from_bits(uint32_t bits) {
  if (bits & kStRange) return SPCONV_ERANGE;
  if (bits & kStDup) return SPCONV_EDUP;
  if (bits & kStCap) return SPCONV_ECAP;
  return SPCONV_OK;
}

int sync_rulebook(spconv_rulebook rb) {
  if (rb->synced) return rb->status;
  DeviceHeader h{};
  if (hipMemcpyAsync(&h, rb->hdr, sizeof(h), hipMemcpyDeviceToHost, rb->stream) != hipSuccess ||
      hipStreamSynchronize(rb->stream) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_EHIP;
  }
  if (rb->in_count) {
    int64_t n_in = 0;
    if (hipMemcpyAsync(&n_in, rb->n_in_dev, sizeof(n_in), hipMemcpyDeviceToHost, rb->stream) !=
            hipSuccess ||
        hipStreamSynchronize(rb->stream) != hipSuccess) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
    rb->n_in = n_in;
  }
  rb->synced = true;
  rb->status = status_from_bits(h.status);
  rb->n_out = h.n_out;
  return rb->status;
}

std::mutex g_alloc_mu;
Allocator g_alloc;                 // the allocator new builds take

// Record that work reading rb was enqueued on `stream` (after it was
// enqueued).  On the build stream nothing is needed: the release is ordered
// there.  On another stream an event is (re)recorded after the work, for the
// release to wait on; if no event can be made, the stream is drained now.
int note_use(spconv_rulebook rb, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (st == rb->stream) return SPCONV_OK;
  std::lock_guard<std::mutex> lk(rb->uses_mu);
  spconv_rulebook_s::Use* u = nullptr;
  for (auto& e : rb->uses)
    if (e.stream == st) u = &e;
  if (!u) {
    hipEvent_t ev;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) == hipSuccess) {
      rb->uses.push_back({st, ev});
      u = &rb->uses.back();
    }
  }
  if (u && hipEventRecord(u->done, st) == hipSuccess) return SPCONV_OK;
  (void)hipGetLastError();
  if (hipStreamSynchronize(st) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_EHIP;
  }
  return SPCONV_OK;
}

int used_on(spconv_rulebook rb, void* stream, int st) {
  if (st != SPCONV_OK) return st;
  return note_use(rb, stream);
}

void release(spconv_rulebook rb) {
  if (!rb) return;
  // the memory is freed on the build stream, after every other stream's
  // latest work on this book
  for (auto& u : rb->uses) {
    (void)hipStreamWaitEvent(rb->stream, u.done, 0);
    (void)hipEventDestroy(u.done);
  }
  rb->uses.clear();
  if (rb->mem) (void)dev_free(rb, rb->mem, rb->stream);
  (void)hipGetLastError();
  delete rb;
}

}  // namespace

int spc::dev_alloc(spconv_rulebook rb, size_t bytes, hipStream_t st, void** p) {
  *p = nullptr;
  if (rb->al.alloc) {
    *p = rb->al.alloc(bytes, st, rb->al.ctx);
    return *p ? SPCONV_OK : SPCONV_ENOMEM;
  }
  *p = cache_alloc(rb->device, bytes, st);
  return *p ? SPCONV_OK : SPCONV_ENOMEM;
}

int spc::dev_free(spconv_rulebook rb, void* p, hipStream_t st) {
  if (!p) return SPCONV_OK;
  if (rb->al.release) {
    rb->al.release(p, st, rb->al.ctx);
    return SPCONV_OK;
  }
  return cache_free(rb->device, p, st) == SPCONV_OK ? SPCONV_OK : SPCONV_EHIP;
}

extern "C" {

int spconv_set_allocator(void* (*alloc)(size_t, void*, void*),
                         void (*release_fn)(void*, void*, void*), void* ctx) {
  if ((alloc == nullptr) != (release_fn == nullptr)) return SPCONV_EINVAL;
  std::lock_guard<std::mutex> lk(g_alloc_mu);
  g_alloc.alloc = alloc;
  g_alloc.release = release_fn;
  g_alloc.ctx = alloc ? ctx : nullptr;
  return SPCONV_OK;
}

int spconv_release_cached_memory(int64_t* released) {
  const size_t n = cache_release_all();
  if (released) *released = static_cast<int64_t>(n);
  return SPCONV_OK;
}

int spconv_memory_stats(int device, int64_t* in_use, int64_t* cached) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_EHIP;
  }
  if (device < 0 || device >= n) return SPCONV_EINVAL;
  size_t live = 0, idle = 0;
  cache_stats(device, &live, &idle);
  if (in_use) *in_use = static_cast<int64_t>(live);
  if (cached) *cached = static_cast<int64_t>(idle);
  return SPCONV_OK;
}

const char* spconv_status_string(int s) {
  switch (s) {
    case SPCONV_OK: return "ok";
    case SPCONV_EINVAL: return "invalid argument";
    case SPCONV_EDUP: return "duplicate site in the input coordinates";
    case SPCONV_ERANGE: return "coordinate outside the grid";
    case SPCONV_ENOMEM: return "device allocation failed";
    case SPCONV_ECAP: return "hash table full";
    case SPCONV_EHIP: return "HIP runtime error";
    case SPCONV_ESCRATCH: return "request exceeds the library's fixed scratch array";
    default: return "unknown status";
  }
}

}  // extern "C"

// Internal status: a book on another book's outputs cannot take the grid
// path; the caller reads the count on the host and builds normally.
constexpr int kNeedHostCount = 2;

// The build behind both entry points.  in_count (device) set: rows [0, N)
// of coords are a bound and only the first *in_count exist.
static int build_impl(int kind, int D, const int32_t* coords, int64_t N,
                      const int64_t* in_count, const int32_t* spatial_size, const int32_t* f,
                      const int32_t* s, unsigned flags, void* stream, spconv_rulebook* out) {
  if (!out) return SPCONV_EINVAL;
  *out = nullptr;
  if (kind != SPCONV_VSC && kind != SPCONV_SC) return SPCONV_EINVAL;
  if (D < 2 || D > kMaxD || N < 0 || N >= 0x7fffffffll) return SPCONV_EINVAL;
  if (N > 0 && (!coords || (reinterpret_cast<uintptr_t>(coords) & 3))) return SPCONV_EINVAL;
  if (!spatial_size || !f || !s ||
      (flags & ~static_cast<unsigned>(SPCONV_BUILD_ASYNC | SPCONV_BUILD_TRANSPOSE)))
    return SPCONV_EINVAL;
  const bool transpose = (flags & SPCONV_BUILD_TRANSPOSE) != 0;
  if (transpose && kind != SPCONV_SC) return SPCONV_EINVAL;
  if (f[0] != 1 || s[0] != 1) return SPCONV_EINVAL;
  int64_t K = 1;
  for (int j = 0; j < D; ++j) {
    if (spatial_size[j] < 1 || spatial_size[j] > 65535 || f[j] < 1 || s[j] < 1)
      return SPCONV_EINVAL;
    if (kind == SPCONV_VSC && (f[j] % 2 != 1 || s[j] != 1)) return SPCONV_EINVAL;
    K *= f[j];
    if (K > kMaxK) return SPCONV_EINVAL;
  }

  auto* rb = new (std::nothrow) spconv_rulebook_s();
  if (!rb) return SPCONV_ENOMEM;
  rb->kind = kind;
  rb->D = D;
  rb->n_in = N;
  rb->n_in_bound = N;
  rb->in_count = in_count;
  rb->K = K;
  rb->stream = static_cast<hipStream_t>(stream);
  {
    std::lock_guard<std::mutex> lk(g_alloc_mu);
    rb->al = g_alloc;
  }
  (void)hipGetDevice(&rb->device);
  uint64_t cells = 1, fan = 1;
  for (int j = 0; j < D; ++j) {
    rb->size[j] = spatial_size[j];
    rb->f[j] = f[j];
    rb->s[j] = s[j];
    if (kind == SPCONV_VSC) {
      rb->out_size[j] = spatial_size[j];
    } else {
      rb->out_size[j] = spatial_size[j] >= f[j] ? (spatial_size[j] - f[j]) / s[j] + 1 : 0;
      cells *= static_cast<uint64_t>(rb->out_size[j]);
      fan *= static_cast<uint64_t>((f[j] + s[j] - 1) / s[j]);
    }
  }
  if (kind == SPCONV_VSC) {
    rb->n_cap = N;
  } else {
    // The SC output set is ranked through a bitmap over the output grid.
    if (cells > (1ull << 32)) {
      delete rb;
      return SPCONV_EINVAL;
    }
    const uint64_t bound = static_cast<uint64_t>(N) * fan;
    rb->n_cap = static_cast<int64_t>(bound < cells ? bound : cells);
    if (rb->n_cap >= 0x7fffffffll) {
      delete rb;
      return SPCONV_EINVAL;
    }
  }
  rb->nblk = (rb->n_cap + kBlock - 1) / kBlock;
  rb->gstride = rb->nblk * kBlock;
  if (in_count && N > 0 && !grid_build(rb)) {
    delete rb;
    return kNeedHostCount;
  }

  // One persistent allocation: header, output sites, gather map, counts,
  // offsets and the pair lists (sized for the worst case K * n_cap so the
  // build never waits for the device to learn k_i).
  const size_t n_cap = static_cast<size_t>(rb->n_cap);
  const size_t Kz = static_cast<size_t>(K);
  size_t bytes = 256;
  bytes += align_up(n_cap * D * 4, 256);
  bytes += align_up(Kz * static_cast<size_t>(rb->gstride) * 4, 256);
  bytes += align_up(Kz * static_cast<size_t>(rb->nblk) * 4 * 2, 256);
  bytes += align_up(Kz * 8, 256);
  bytes += align_up((Kz + 1) * 8, 256);
  bytes += align_up(Kz * n_cap * 8, 256);
  bytes += align_up(n_cap * 4, 256);
  const size_t tbytes = transpose ? transpose_bytes(N, K) : 0;
  bytes += tbytes;
  if (dev_alloc(rb, bytes, rb->stream, &rb->mem) != SPCONV_OK) {
    delete rb;
    return SPCONV_ENOMEM;
  }
  rb->mem_bytes = bytes;
  char* p = static_cast<char*>(rb->mem);
  size_t off = 0;
  auto take = [&](size_t b) {
    char* q = p + off;
    off += align_up(b, 256);
    return q;
  };
  rb->hdr = reinterpret_cast<DeviceHeader*>(take(256));
  rb->n_in_dev = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(rb->hdr) + 128);
  // (with rows, the input scatter of the grid build copies the count)
  if (in_count && N == 0) copy_in_count(rb);
  rb->out_coords = reinterpret_cast<int32_t*>(take(n_cap * D * 4));
  rb->gmap = reinterpret_cast<int32_t*>(take(Kz * static_cast<size_t>(rb->gstride) * 4));
  rb->blk_cnt = reinterpret_cast<int32_t*>(take(Kz * static_cast<size_t>(rb->nblk) * 4 * 2));
  rb->wpre = reinterpret_cast<uint32_t*>(rb->blk_cnt + Kz * static_cast<size_t>(rb->nblk));
  rb->totals = reinterpret_cast<int64_t*>(take(Kz * 8));
  rb->pair_off = reinterpret_cast<int64_t*>(take((Kz + 1) * 8));
  rb->pairs = reinterpret_cast<int32_t*>(take(Kz * n_cap * 8));
  rb->perm = reinterpret_cast<int32_t*>(take(n_cap * 4));
  char* tmem = transpose ? take(tbytes) : nullptr;

  int st = kind == SPCONV_VSC ? build_vsc(rb, coords) : build_sc(rb, coords);
  if (st == SPCONV_OK && transpose) st = build_transpose(rb, coords, tmem);
  if (st != SPCONV_OK) {
    release(rb);
    return st;
  }
  if (!(flags & SPCONV_BUILD_ASYNC)) {
    st = sync_rulebook(rb);
    if (st != SPCONV_OK) {
      release(rb);
      return st;
    }
  }
  *out = rb;
  return SPCONV_OK;
}

extern "C" {

int spconv_build_rulebook(int kind, int D, const int32_t* coords, int64_t N,
                          const int32_t* spatial_size, const int32_t* f, const int32_t* s,
                          unsigned flags, void* stream, spconv_rulebook* out) {
  return build_impl(kind, D, coords, N, nullptr, spatial_size, f, s, flags, stream, out);
}

int spconv_build_rulebook_on(spconv_rulebook parent, int kind, const int32_t* f, const int32_t* s,
                             unsigned flags, void* stream, spconv_rulebook* out) {
  if (!out) return SPCONV_EINVAL;
  *out = nullptr;
  if (!parent || parent->kind != SPCONV_SC || (flags & SPCONV_BUILD_TRANSPOSE))
    return SPCONV_EINVAL;
  const int st = build_impl(kind, parent->D, parent->out_coords, parent->n_cap,
                            &parent->hdr->n_out, parent->out_size, f, s, flags, stream, out);
  if (st != kNeedHostCount) return used_on(parent, stream, st);
  // the hash-table path needs the count on the host: read it, build normally
  int64_t n = 0;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(&n, &parent->hdr->n_out, sizeof(n), hipMemcpyDeviceToHost, hs) !=
          hipSuccess ||
      hipStreamSynchronize(hs) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_EHIP;
  }
  return used_on(parent, stream,
                 build_impl(kind, parent->D, parent->out_coords, n, nullptr, parent->out_size,
                            f, s, flags, stream, out));
}

int spconv_rulebook_bounds(spconv_rulebook rb, int64_t* n_in_bound, int64_t* n_out_bound) {
  if (!rb) return SPCONV_EINVAL;
  if (n_in_bound) *n_in_bound = rb->n_in_bound;
  if (n_out_bound) *n_out_bound = rb->n_cap;
  return SPCONV_OK;
}

int spconv_rulebook_status(spconv_rulebook rb) {
  if (!rb) return SPCONV_EINVAL;
  return sync_rulebook(rb);
}

int spconv_rulebook_query(spconv_rulebook rb, int64_t* n_in, int64_t* n_out, int64_t* K,
                          int32_t* out_spatial_size, int64_t* pair_off) {
  if (!rb) return SPCONV_EINVAL;
  const int st = sync_rulebook(rb);
  if (st == SPCONV_EHIP) return st;
  if (n_in) *n_in = rb->n_in;
  if (n_out) *n_out = rb->n_out;
  if (K) *K = rb->K;
  if (out_spatial_size)
    for (int j = 0; j < rb->D; ++j) out_spatial_size[j] = rb->out_size[j];
  if (pair_off) {
    if (hipMemcpyAsync(pair_off, rb->pair_off, (rb->K + 1) * sizeof(int64_t),
                       hipMemcpyDeviceToHost, rb->stream) != hipSuccess ||
        hipStreamSynchronize(rb->stream) != hipSuccess) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
  }
  return st;
}

int spconv_rulebook_export(spconv_rulebook rb, int32_t* out_coords, int32_t* pairs,
                           void* stream) {
  if (!rb) return SPCONV_EINVAL;
  int st = sync_rulebook(rb);
  if (st != SPCONV_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (out_coords && rb->n_out > 0) {
    if (hipMemcpyAsync(out_coords, rb->out_coords, rb->n_out * rb->D * sizeof(int32_t),
                       hipMemcpyDeviceToDevice, s) != hipSuccess) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
  }
  if (pairs) {
    int64_t total = 0;
    if (hipMemcpyAsync(&total, rb->pair_off + rb->K, sizeof(int64_t), hipMemcpyDeviceToHost,
                       rb->stream) != hipSuccess ||
        hipStreamSynchronize(rb->stream) != hipSuccess) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
    if (total > 0 &&
        hipMemcpyAsync(pairs, rb->pairs, total * 2 * sizeof(int32_t), hipMemcpyDeviceToDevice,
                       s) != hipSuccess) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
  }
  return note_use(rb, stream);
}

int spconv_rulebook_out_coords(spconv_rulebook rb, const int32_t** coords) {
  if (!rb || !coords) return SPCONV_EINVAL;
  *coords = rb->out_coords;
  return SPCONV_OK;
}

// Argument checks shared by the forward entry points; with check_only nothing
// is launched.
// Output rows of a book as far as the host knows them: the count once the
// book is synchronised, its bound before.  A pointer to rows that turn out to
// be none may be NULL.
static int64_t out_rows(spconv_rulebook rb) { return rb->synced ? rb->n_out : rb->n_cap; }

static int forward_common(spconv_rulebook rb, int kind, int in_dt, const void* x, const void* w,
                          const float* bias, int out_dt, void* y, int C_in, int C_out,
                          void* stream, bool check_only = false) {
  if (!rb || rb->kind != kind) return SPCONV_EINVAL;
  if ((in_dt != SPCONV_F32 && in_dt != SPCONV_BF16) ||
      (out_dt != SPCONV_F32 && out_dt != SPCONV_BF16))
    return SPCONV_EINVAL;
  if (C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  if (out_rows(rb) > 0 && (!y || !w || (rb->n_in > 0 && !x))) return SPCONV_EINVAL;
  const uintptr_t al = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w) |
                       reinterpret_cast<uintptr_t>(y);
  if ((al & 15) || (reinterpret_cast<uintptr_t>(bias) & 3)) return SPCONV_EINVAL;
  if (check_only) return SPCONV_OK;
  return used_on(rb, stream, forward(rb, in_dt, x, w, bias, out_dt, y, C_in, C_out,
                                     static_cast<hipStream_t>(stream)));
}

int spconv_vsc_forward(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                       const float* bias, int out_dt, void* y, int C_in, int C_out,
                       void* stream) {
  return forward_common(rb, SPCONV_VSC, in_dt, x, w, bias, out_dt, y, C_in, C_out, stream);
}

int spconv_sc_forward(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                      const float* bias, int out_dt, void* y, int C_in, int C_out,
                      void* stream) {
  return forward_common(rb, SPCONV_SC, in_dt, x, w, bias, out_dt, y, C_in, C_out, stream);
}

int spconv_forward_fused(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                         const float* scale, const float* shift, const void* residual,
                         int relu, int out_dt, void* y, int C_in, int C_out, void* stream) {
  if (!rb || (rb->kind != SPCONV_VSC && rb->kind != SPCONV_SC)) return SPCONV_EINVAL;
  if (relu != 0 && relu != 1) return SPCONV_EINVAL;
  if ((reinterpret_cast<uintptr_t>(scale) & 3) || (reinterpret_cast<uintptr_t>(residual) & 15))
    return SPCONV_EINVAL;
  // the residual may be y itself, but no other overlap (checked once the
  // output row count is known on the host)
  if (residual && residual != y && y && rb->synced && rb->n_out > 0 && C_out > 0) {
    const size_t bytes = static_cast<size_t>(rb->n_out) * C_out * (out_dt == SPCONV_BF16 ? 2 : 4);
    const uintptr_t r0 = reinterpret_cast<uintptr_t>(residual), y0 = reinterpret_cast<uintptr_t>(y);
    if (r0 < y0 + bytes && y0 < r0 + bytes) return SPCONV_EINVAL;
  }
  const int st = forward_common(rb, rb->kind, in_dt, x, w, shift, out_dt, y, C_in, C_out,
                                nullptr, /*check_only=*/true);
  if (st != SPCONV_OK) return st;
  Epilogue e;
  e.scale = scale;
  e.res = residual;
  e.relu = relu;
  return used_on(rb, stream, forward_view(view_of(rb), 0, in_dt, x, w, shift, out_dt, y, C_in,
                                          C_out, static_cast<hipStream_t>(stream), e));
}

static bool dtype_ok(int dt) { return dt == SPCONV_F32 || dt == SPCONV_BF16; }
static bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

int spconv_pool_forward(spconv_rulebook rb, int mode, int dt, const void* x, void* y, int C,
                        void* stream) {
  if (!rb || rb->kind != SPCONV_SC || !dtype_ok(dt) || C < 1) return SPCONV_EINVAL;
  if (mode != SPCONV_POOL_MAX && mode != SPCONV_POOL_AVG) return SPCONV_EINVAL;
  if (out_rows(rb) > 0 && (!y || (rb->n_in > 0 && !x))) return SPCONV_EINVAL;
  if (misaligned(x) || misaligned(y)) return SPCONV_EINVAL;
  return used_on(rb, stream, pool_forward(rb, mode, dt, x, y, C, static_cast<hipStream_t>(stream)));
}

int spconv_dc_forward(spconv_rulebook rb, int in_dt, const void* x, const void* w,
                      const float* bias, int out_dt, void* y, int C_in, int C_out,
                      void* stream) {
  if (!rb || rb->kind != SPCONV_SC || !rb->t_gmap) return SPCONV_EINVAL;
  if (!dtype_ok(in_dt) || !dtype_ok(out_dt) || C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  if (rb->n_in > 0 && (!y || !w || (out_rows(rb) > 0 && !x))) return SPCONV_EINVAL;
  if (misaligned(x) || misaligned(w) || misaligned(y) ||
      (reinterpret_cast<uintptr_t>(bias) & 3))
    return SPCONV_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (rb->t_single && rb->n_in > 0) {
    const int r = transpose_single(rb, 0, in_dt, x, w, bias, out_dt, y, C_in, C_out, st);
    if (r != kNotSingle) return used_on(rb, stream, r);
  }
  return used_on(rb, stream, forward_view(transpose_view(rb), 0, in_dt, x, w, bias, out_dt, y,
                                          C_in, C_out, st));
}

// The book, view and weight mode an input gradient runs on.
static int data_grad_view(spconv_rulebook rb, int op, FwdView* v, int* wmode) {
  if (!rb) return SPCONV_EINVAL;
  switch (op) {
    case SPCONV_OP_VSC:
      if (rb->kind != SPCONV_VSC) return SPCONV_EINVAL;
      *v = view_of(rb);              // VSC pairs are symmetric: flip the offsets
      *wmode = 1;
      return SPCONV_OK;
    case SPCONV_OP_SC:
      if (rb->kind != SPCONV_SC || !rb->t_gmap) return SPCONV_EINVAL;
      *v = transpose_view(rb);       // SC pairs reversed
      *wmode = 2;
      return SPCONV_OK;
    case SPCONV_OP_DC:
      if (rb->kind != SPCONV_SC) return SPCONV_EINVAL;
      *v = view_of(rb);              // DC's reversed pairs reversed again
      *wmode = 2;
      return SPCONV_OK;
    default:
      return SPCONV_EINVAL;
  }
}

int spconv_backward_data(spconv_rulebook rb, int op, int dt, const void* dy, const void* w,
                         int out_dt, void* dx, int C_in, int C_out, void* stream) {
  FwdView v;
  int wmode = 0;
  const int vs = data_grad_view(rb, op, &v, &wmode);
  if (vs != SPCONV_OK) return vs;
  if (!dtype_ok(dt) || !dtype_ok(out_dt) || C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  // rows of dx and dy: VSC both n_in; SC dx n_in, dy n_out; DC the reverse
  const int64_t dst = op == SPCONV_OP_DC ? out_rows(rb) : rb->n_in;
  const int64_t src = op == SPCONV_OP_SC ? out_rows(rb) : rb->n_in;
  if (dst > 0 && (!dx || !w || (src > 0 && !dy))) return SPCONV_EINVAL;
  if (misaligned(dy) || misaligned(w) || misaligned(dx)) return SPCONV_EINVAL;
  // the kernels' input channels are the layer's output channels
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (op == SPCONV_OP_SC && rb->t_single && rb->n_in > 0) {
    const int r = transpose_single(rb, wmode, dt, dy, w, nullptr, out_dt, dx, C_out, C_in, st);
    if (r != kNotSingle) return used_on(rb, stream, r);
  }
  return used_on(rb, stream, forward_view(v, wmode, dt, dy, w, nullptr, out_dt, dx, C_out, C_in,
                                          st));
}

int spconv_backward_weight_workspace(spconv_rulebook rb, int op, int C_in, int C_out,
                                     size_t* bytes) {
  if (!rb || !bytes || C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  if (op == SPCONV_OP_DC ? rb->kind != SPCONV_SC : op != rb->kind) return SPCONV_EINVAL;
  *bytes = backward_weight_workspace(rb, C_in, C_out, op);
  return SPCONV_OK;
}

int spconv_backward_weight(spconv_rulebook rb, int op, int dt, const void* x, const void* dy,
                           float* dw, float* db, int C_in, int C_out, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (!rb || C_in < 1 || C_out < 1 || !dtype_ok(dt) || !dw) return SPCONV_EINVAL;
  if (op == SPCONV_OP_DC ? rb->kind != SPCONV_SC : op != rb->kind) return SPCONV_EINVAL;
  if (!workspace || workspace_bytes < backward_weight_workspace(rb, C_in, C_out, op))
    return SPCONV_EINVAL;
  if (misaligned(x) || misaligned(dy) || misaligned(workspace) ||
      (reinterpret_cast<uintptr_t>(dw) & 3) || (reinterpret_cast<uintptr_t>(db) & 3))
    return SPCONV_EINVAL;
  const int st = sync_rulebook(rb);    // the bias gradient needs n_out on the host
  if (st != SPCONV_OK) return st;
  // rows of x and dy: VSC both n_in; SC x n_in, dy n_out; DC the reverse
  const int64_t xr = op == SPCONV_OP_DC ? rb->n_out : rb->n_in;
  const int64_t gr = op == SPCONV_OP_SC ? rb->n_out : rb->n_in;
  if ((xr > 0 && !x) || (gr > 0 && !dy)) return SPCONV_EINVAL;
  return used_on(rb, stream, backward_weight(rb, op, dt, x, dy, dw, db, C_in, C_out, workspace,
                                             static_cast<hipStream_t>(stream)));
}

void spconv_rulebook_destroy(spconv_rulebook rb) { release(rb); }

}  // extern "C"
