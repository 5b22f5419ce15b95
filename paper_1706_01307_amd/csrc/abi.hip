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

// Keep freed stream-ordered memory in the device's default pool, so that
// rule books rebuilt every step reuse it instead of returning it to the
// driver.
void keep_pool_memory(int dev) {
  static std::mutex mu;
  static bool done[64] = {};
  std::lock_guard<std::mutex> lk(mu);
  if (dev < 0 || dev >= 64 || done[dev]) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t thr = ~0ull;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
  }
  (void)hipGetLastError();
  done[dev] = true;
}

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
  rb->synced = true;
  rb->status = status_from_bits(h.status);
  rb->n_out = h.n_out;
  return rb->status;
}

void release(spconv_rulebook rb) {
  if (!rb) return;
  if (rb->mem) (void)hipFreeAsync(rb->mem, rb->stream);
  (void)hipGetLastError();
  delete rb;
}

}  // namespace

extern "C" {

const char* spconv_status_string(int s) {
  switch (s) {
    case SPCONV_OK: return "ok";
    case SPCONV_EINVAL: return "invalid argument";
    case SPCONV_EDUP: return "duplicate site in the input coordinates";
    case SPCONV_ERANGE: return "coordinate outside the grid";
    case SPCONV_ENOMEM: return "device allocation failed";
    case SPCONV_ECAP: return "hash table full";
    case SPCONV_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int spconv_build_rulebook(int kind, int D, const int32_t* coords, int64_t N,
                          const int32_t* spatial_size, const int32_t* f, const int32_t* s,
                          unsigned flags, void* stream, spconv_rulebook* out) {
  if (!out) return SPCONV_EINVAL;
  *out = nullptr;
  if (kind != SPCONV_VSC && kind != SPCONV_SC) return SPCONV_EINVAL;
  if (D < 2 || D > kMaxD || N < 0 || N >= 0x7fffffffll) return SPCONV_EINVAL;
  if (N > 0 && (!coords || (reinterpret_cast<uintptr_t>(coords) & 3))) return SPCONV_EINVAL;
  if (!spatial_size || !f || !s || (flags & ~static_cast<unsigned>(SPCONV_BUILD_ASYNC)))
    return SPCONV_EINVAL;
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
  rb->K = K;
  rb->stream = static_cast<hipStream_t>(stream);
  (void)hipGetDevice(&rb->device);
  keep_pool_memory(rb->device);
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
  if (hipMallocAsync(&rb->mem, bytes, rb->stream) != hipSuccess) {
    (void)hipGetLastError();
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
  rb->out_coords = reinterpret_cast<int32_t*>(take(n_cap * D * 4));
  rb->gmap = reinterpret_cast<int32_t*>(take(Kz * static_cast<size_t>(rb->gstride) * 4));
  rb->blk_cnt = reinterpret_cast<int32_t*>(take(Kz * static_cast<size_t>(rb->nblk) * 4 * 2));
  rb->wpre = reinterpret_cast<uint32_t*>(rb->blk_cnt + Kz * static_cast<size_t>(rb->nblk));
  rb->totals = reinterpret_cast<int64_t*>(take(Kz * 8));
  rb->pair_off = reinterpret_cast<int64_t*>(take((Kz + 1) * 8));
  rb->pairs = reinterpret_cast<int32_t*>(take(Kz * n_cap * 8));
  rb->perm = reinterpret_cast<int32_t*>(take(n_cap * 4));

  int st = kind == SPCONV_VSC ? build_vsc(rb, coords) : build_sc(rb, coords);
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
  return SPCONV_OK;
}

int spconv_rulebook_out_coords(spconv_rulebook rb, const int32_t** coords) {
  if (!rb || !coords) return SPCONV_EINVAL;
  *coords = rb->out_coords;
  return SPCONV_OK;
}

static int forward_common(spconv_rulebook rb, int kind, int in_dt, const void* x, const void* w,
                          const float* bias, int out_dt, void* y, int C_in, int C_out,
                          void* stream) {
  if (!rb || rb->kind != kind) return SPCONV_EINVAL;
  if ((in_dt != SPCONV_F32 && in_dt != SPCONV_BF16) ||
      (out_dt != SPCONV_F32 && out_dt != SPCONV_BF16))
    return SPCONV_EINVAL;
  if (C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  if (rb->n_cap > 0 && (!y || !w || (rb->n_in > 0 && !x))) return SPCONV_EINVAL;
  const uintptr_t al = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w) |
                       reinterpret_cast<uintptr_t>(y);
  if ((al & 15) || (reinterpret_cast<uintptr_t>(bias) & 3)) return SPCONV_EINVAL;
  return forward(rb, in_dt, x, w, bias, out_dt, y, C_in, C_out, static_cast<hipStream_t>(stream));
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

void spconv_rulebook_destroy(spconv_rulebook rb) { release(rb); }

}  // extern "C"
