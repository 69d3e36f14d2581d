// Shared device/host definitions of the HIP kernels in libherald.so (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "herald.h"

namespace herald {

// Device-side copy of a KV view (passed by value to kernels).
struct KvView {
  const char *k;
  const char *v;
  int64_t sb, sh, ss;    // strides in elements
  const int32_t *pt;     // page table or nullptr
  int32_t page_shift;    // log2(page_size), paged only
  int32_t max_pages;
  int64_t sp;            // page stride in elements
  const int32_t *lens;   // valid rows per sequence
  int64_t max_len;       // host bound; lens[b] is clamped to it
};

// Valid rows of sequence b, clamped to the host bound of the view.
__device__ __forceinline__ int64_t kv_len(const KvView &kv, int b) {
  const int64_t n = kv.lens[b];
  return n < 0 ? 0 : (n > kv.max_len ? kv.max_len : n);
}

// Writable contiguous view.
struct PoolView {
  char *k;
  char *v;
  int64_t sb, sh, ss;
};

// Element offset of row s of head h of sequence b.
__device__ __forceinline__ int64_t kv_row(const KvView &kv, int b, int h,
                                          int64_t s) {
  if (kv.pt == nullptr) return (int64_t)b * kv.sb + (int64_t)h * kv.sh + s * kv.ss;
  const int64_t page = kv.pt[(int64_t)b * kv.max_pages + (s >> kv.page_shift)];
  return page * kv.sp + (int64_t)h * kv.sh +
         (s & ((1 << kv.page_shift) - 1)) * kv.ss;
}

__device__ __forceinline__ uint4 ldg16(const void *p) {
  return *reinterpret_cast<const uint4 *>(p);
}

// Streaming (non-temporal) 16-byte load: data read once, kept out of the way
// of data that is re-read soon.
__device__ __forceinline__ uint4 ldg16_nt(const void *p) {
  const uint4 *q = reinterpret_cast<const uint4 *>(p);
  uint4 r;
  r.x = __builtin_nontemporal_load(&q->x);
  r.y = __builtin_nontemporal_load(&q->y);
  r.z = __builtin_nontemporal_load(&q->z);
  r.w = __builtin_nontemporal_load(&q->w);
  return r;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

__device__ __forceinline__ int clamp_k(int k, int64_t S, int k_max) {
  int64_t kk = k < 0 ? 0 : k;
  if (kk > S) kk = S;
  if (kk > k_max) kk = k_max;
  return (int)kk;
}

}  // namespace herald

// ---- launchers (host side, defined in the .hip files) -----------------------
namespace herald {

hipError_t launch_gather(const herald_heads &hd, int batch, const KvView &kv,
                         const int32_t *idx, const int32_t *k_per_seq, int k_max,
                         const PoolView &dst, int dst_row0, hipStream_t stream);

struct AttnPlan {
  int M;          // G * block query rows per (b, h)
  int rows_per_wave; // query rows per wave (16 or 32)
  int nwaves;     // waves per pipeline
  int pipes;      // pipelines per workgroup (alternate key tiles)
  int stages;     // LDS stages per pipeline
  int key_tile;   // keys per tile
  int n_mblk;     // row blocks per (b, h)
  int nsplit;     // key splits of this call
  int nsplit_cap; // bound on nsplit for any context up to this one (sizes the workspace)
  int keys_per_split;
  size_t part_o_bytes, part_ml_bytes;
};

AttnPlan attn_plan(const herald_heads &hd, int batch, int block, int64_t max_ctx);

// groups query groups of `block` rows per sequence (q, blk_k/blk_v and out
// hold batch * groups groups); the groups of sequence b share its context and
// each sees only its own block KV.
hipError_t launch_block_attn(const herald_heads &hd, int batch, int block, int groups,
                             const void *q, const KvView &ctx, int64_t max_ctx,
                             const void *blk_k, const void *blk_v, void *out,
                             void *ws, hipStream_t stream);

hipError_t launch_append(const herald_heads &hd, int batch, int block,
                         const void *done_k, const void *done_v,
                         const PoolView &cache, const int32_t *seq_lens,
                         const PoolView *idle, const int32_t *k_next, int k_max,
                         int64_t cache_cap, hipStream_t stream);

hipError_t launch_bump(int batch, int block, int32_t *seq_lens, int32_t *n_idle,
                       const int32_t *k_next, int k_max, hipStream_t stream);

}  // namespace herald
