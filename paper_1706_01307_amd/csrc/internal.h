// Internal declarations of the gfx950 sparse-convolution library.
//
// Everything in here is device-side building blocks shared by the rule-book
// and forward translation units, plus the host-side rule-book object.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "spconv.h"
#include "forward_types.h"

namespace spc {

// ---------------------------------------------------------------------------
// Status bits written by device kernels (OR-ed into one word).
// ---------------------------------------------------------------------------
enum : uint32_t { kStRange = 1u, kStDup = 2u, kStCap = 4u };

constexpr int kMaxD = 4;
constexpr int kMaxK = 1024;          // filter offsets per layer
constexpr uint64_t kEmpty = ~0ull;   // empty hash slot
constexpr int kBlock = 256;          // rows per rule-book block (4 waves)


// ---------------------------------------------------------------------------
// Order-preserving site codec: coordinate j occupies `bits[j]` bits at
// `shift[j]`, coordinate 0 (sample) in the high bits, so integer order of
// keys is lexicographic order of sites.
// ---------------------------------------------------------------------------
struct Codec {
  int D;
  int kbits;                 // total key bits
  int shift[kMaxD];
  uint32_t fmask[kMaxD];
  int32_t size[kMaxD];
};

__host__ __device__ inline uint64_t pack_site(const Codec& c, const int32_t* x) {
  uint64_t k = 0;
  for (int j = 0; j < c.D; ++j) k |= static_cast<uint64_t>(x[j]) << c.shift[j];
  return k;
}

__host__ __device__ inline void unpack_site(const Codec& c, uint64_t k, int32_t* x) {
  for (int j = 0; j < c.D; ++j)
    x[j] = static_cast<int32_t>((k >> c.shift[j]) & c.fmask[j]);
}

// ---------------------------------------------------------------------------
// Open-addressing hash table of sites -> rows.  Slots are grouped in
// buckets of 4 (32 bytes) and buckets in lines of 4 (128 bytes, one cache
// line).  The home line of a site is a hash of its 2x2(x2) brick, i.e. of the
// key with the lowest bit of every spatial coordinate cleared; the bucket
// inside the line is picked by two of those low bits.  So the sites of one
// brick share a cache line, and the 3^d neighbours of a site fall in at most
// 2^d lines, which neighbouring sites share as well.  A lookup reads its home
// bucket and moves on (linearly) only when all 4 slots are taken.
// Packed layout: slot = key << rbits | row (one 64-bit word, one CAS per
// insert).  Wide layout (when key bits + row bits exceed 64): key words in
// `slots`, rows in `vals`.
// ---------------------------------------------------------------------------
struct Table {
  uint64_t* slots;
  int32_t* vals;       // wide layout only
  uint64_t nbuckets;   // power of two
  int rbits;           // packed layout: bits of the row field
  uint64_t brick_mask; // key bits that identify the brick
  uint64_t lmask1;     // key bit selecting bucket bit 1 (0: none)
  uint64_t lmask0;     // key bit selecting bucket bit 0 (0: none)
  int line_shift;      // log2(buckets per line): 2 = brick lines, 0 = plain hash
};

__device__ __forceinline__ uint64_t mix64(uint64_t k) {
  // 64-bit finaliser (xor-shift / multiply avalanche).
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

__device__ __forceinline__ uint64_t home_bucket(const Table& t, uint64_t key) {
  const uint64_t nlines = (t.nbuckets >> t.line_shift) ? (t.nbuckets >> t.line_shift) : 1;
  const uint64_t line = mix64(key & t.brick_mask) & (nlines - 1);
  const uint64_t local = ((key & t.lmask1) ? 2u : 0u) | ((key & t.lmask0) ? 1u : 0u);
  return ((line << t.line_shift) | local) & (t.nbuckets - 1);
}

// Match one bucket (4 slots already loaded) against `key`.
// Returns the row (>= 0), -1 if the key is absent (an empty slot was seen),
// or -2 if the bucket is full without the key (continue to the next bucket).
// Slots fill in order, so the first empty slot ends the search.  Written as a
// select chain over all 4 slots (last slot first): every loaded slot is used
// on every path, so the compiler keeps the whole bucket load unconditional.
template <bool WIDE>
__device__ __forceinline__ int32_t match_bucket(const Table& t, uint64_t b,
                                                const uint64_t s[4], uint64_t key) {
  int32_t res = -2;
#pragma unroll
  for (int j = 3; j >= 0; --j) {
    const bool empty = s[j] == kEmpty;
    bool hit;
    int32_t row;
    if (WIDE) {
      hit = !empty && s[j] == key;
      row = hit ? t.vals[4 * b + j] : 0;
    } else {
      hit = !empty && (s[j] >> t.rbits) == key;
      row = static_cast<int32_t>(s[j] & ((1ull << t.rbits) - 1));
    }
    res = hit ? row : (empty ? -1 : res);
  }
  return res;
}

__device__ __forceinline__ void load_bucket(const Table& t, uint64_t b, uint64_t s[4]) {
  const ulonglong2* p = reinterpret_cast<const ulonglong2*>(t.slots + 4 * b);
  ulonglong2 a = p[0], c = p[1];
  s[0] = a.x; s[1] = a.y; s[2] = c.x; s[3] = c.y;
}

// Slow path of a lookup: continue probing after bucket `b` was full.
template <bool WIDE>
__device__ __noinline__ int32_t find_from(const Table& t, uint64_t b, uint64_t key) {
  for (uint64_t p = 1; p < t.nbuckets; ++p) {
    b = (b + 1) & (t.nbuckets - 1);
    uint64_t s[4];
    load_bucket(t, b, s);
    int32_t r = match_bucket<WIDE>(t, b, s, key);
    if (r != -2) return r;
  }
  return -1;
}

}  // namespace spc

// ---------------------------------------------------------------------------
// Host-side rule book.
// ---------------------------------------------------------------------------
namespace spc {
// Where a rule book's device memory comes from: a registered allocator
// (spconv_set_allocator) or, with both functions NULL, the library's block
// cache.  Each rule book keeps the one it was built with.
struct Allocator {
  void* (*alloc)(size_t, void*, void*) = nullptr;
  void (*release)(void*, void*, void*) = nullptr;
  void* ctx = nullptr;
};
}  // namespace spc

struct spconv_rulebook_s {
  int kind;
  int D;
  int device;
  int64_t n_in;                // input rows (a bound until synchronised, for a book
                               // built on another book's outputs)
  int64_t n_in_bound;          // input rows the buffers are sized for
  int64_t n_cap;               // output rows the buffers are sized for
  // A book built on another SC book's output sites: the input row count is
  // that book's device-side output count (read during the build only), and
  // a copy of it lives in this book's header block (n_in_dev).
  const int64_t* in_count = nullptr;
  int64_t* n_in_dev = nullptr;
  int64_t K;
  int32_t size[spc::kMaxD], f[spc::kMaxD], s[spc::kMaxD], out_size[spc::kMaxD];
  hipStream_t stream;          // build stream (owns the allocation)
  spc::Allocator al;           // the allocator the book was built with (and releases through)
  void* mem;                   // one stream-ordered allocation
  size_t mem_bytes;
  // carved device pointers
  spc::DeviceHeader* hdr;
  int32_t* out_coords;         // [n_cap][D]
  int32_t* gmap;               // [K][gstride] 1 + input row per (offset, schedule position); 0 = none
  int64_t gstride;             // gather-map row length: nblk * kBlock (entries past n_out are 0)
  int32_t* blk_cnt;            // [K][nblk] per-block pair counts, then bases
  uint32_t* wpre;              // [K][nblk] per-wave prefixes inside a block (bytes)
  int64_t* totals;             // [K] k_i
  int64_t* pair_off;           // [K+1]
  int32_t* pairs;              // [K * n_cap][2]
  int32_t* perm;               // [n_cap] schedule: output rows in Z-order of their sites
  int64_t nblk;                // ceil(n_cap / kBlock)
  // transposed rule book (SC built with SPCONV_BUILD_TRANSPOSE), or NULL:
  // the SC input rows ordered by offset class, and for every (offset, position
  // in that order) 1 + the SC output row paired with that input row
  spc::DeviceHeader* t_hdr;    // n_out = n_in
  int32_t* t_perm;             // [n_in]
  int32_t* t_gmap;             // [K][t_gstride]
  int64_t t_gstride;
  // f = s: R_i also split into its two columns, each offset's run padded to
  // whole chunks of kSegRows positions (padding: source 0, destination -1)
  bool t_single;
  int64_t t_npad_cap;          // bound on the padded length (sum k + K kSegRows)
  int32_t* t_src;              // [t_npad_cap] 1 + SC output row
  int32_t* t_dst;              // [t_npad_cap] SC input row, -1 = padding
  int32_t* t_seg;              // [t_npad_cap / kSegRows] offset of every chunk
  int32_t* t_chunk_off;        // [K + 1] first chunk of every offset
  spc::DeviceHeader* t_hdrs;   // [K] n_out = k_i; [K] (one more) n_out = padded length
  std::vector<int64_t> h_pair_off;   // host copy of pair_off, filled on first use
  // Streams other than the build stream that work reading this book was
  // enqueued on, each with an event recorded after its latest such work:
  // the release makes the build stream wait on all of them before the
  // memory goes back to the allocator.
  struct Use {
    hipStream_t stream;
    hipEvent_t done;
  };
  std::vector<Use> uses;
  std::mutex uses_mu;
  // host state after synchronisation
  bool synced;
  int status;
  int64_t n_out;
};

namespace spc {

// The library's default allocator (blockcache.hip): blocks of device `dev`
// handed out on, and given back on, a stream; reuse is ordered by events.
// cache_alloc returns nullptr when the device has no memory left;
// cache_free: SPCONV_OK, SPCONV_EINVAL (not a cache block) or SPCONV_EHIP.
void* cache_alloc(int dev, size_t bytes, hipStream_t st);
int cache_free(int dev, void* p, hipStream_t st);
size_t cache_release_all();      // frees the idle blocks of every device
void cache_stats(int dev, size_t* live_bytes, size_t* idle_bytes);

// Stream-ordered device memory through the rule book's allocator.
// dev_alloc: SPCONV_OK or SPCONV_ENOMEM; dev_free: SPCONV_OK or SPCONV_EHIP.
int dev_alloc(spconv_rulebook rb, size_t bytes, hipStream_t st, void** p);
int dev_free(spconv_rulebook rb, void* p, hipStream_t st);

// Launchers (rulebook.hip).  All asynchronous on rb->stream.
int build_vsc(spconv_rulebook rb, const int32_t* coords);
// Whether the build of this book takes the dense-grid path (the one that can
// take a device-side input count).
bool grid_build(spconv_rulebook rb);
// Enqueue the copy of *rb->in_count into rb->n_in_dev.
void copy_in_count(spconv_rulebook rb);
int build_sc(spconv_rulebook rb, const int32_t* coords);

// Radix sort (sort.hip).
size_t radix_sort_scratch_bytes(int64_t n_cap);
bool radix_sort_pairs(uint64_t* keys, int32_t* vals, uint64_t* keys_tmp, int32_t* vals_tmp,
                      const DeviceHeader* hdr, int64_t n_cap, int key_bits, void* scratch,
                      hipStream_t stream, int lo_bit = 0);
int radix_sort_passes(int key_bits, int lo_bit);

FwdView view_of(spconv_rulebook rb);
// wmode 0: W^i = w[i] ([K][C_in][C_out]); 1: w[K-1-i]^T; 2: w[i]^T (w given
// as [K][C_out][C_in] of the layer whose gradient this is).
int forward_view(const FwdView& v, int wmode, int in_dt, const void* x, const void* w,
                 const float* bias, int out_dt, void* y, int C_in, int C_out,
                 hipStream_t stream, const Epilogue& epi = Epilogue{});
int forward(spconv_rulebook rb, int in_dt, const void* x, const void* w,
            const float* bias, int out_dt, void* y, int C_in, int C_out,
            hipStream_t stream);

// Pooling, transposed rule book, weight gradients (ops.hip).
int pool_forward(spconv_rulebook rb, int mode, int dt, const void* x, void* y, int C,
                 hipStream_t stream);
size_t transpose_bytes(int64_t n_in, int64_t K);
int build_transpose(spconv_rulebook rb, const int32_t* coords, char* mem);
FwdView transpose_view(spconv_rulebook rb);
constexpr int kNotSingle = 1;
int transpose_single(spconv_rulebook rb, int wmode, int in_dt, const void* x, const void* w,
                     const float* bias, int out_dt, void* y, int C_in, int C_out,
                     hipStream_t st);
size_t backward_weight_workspace(spconv_rulebook rb, int C_in, int C_out, int op);
int backward_weight(spconv_rulebook rb, int op, int dt, const void* x, const void* dy, float* dw,
                    float* db, int C_in, int C_out, void* ws, hipStream_t stream);

// Host helpers (abi.cpp).
Codec make_codec(int D, const int32_t* size);
inline int bitlen(uint64_t v) { int b = 0; while (v) { ++b; v >>= 1; } return b; }

}  // namespace spc
