// Block-boundary kernels of the two-stream pipeline (sec. IV-B.2 of the
// paper, steps 5-6 of the main stream): the completed block's KV is appended
// to the prefix cache and to the tail of the pool that the next block will
// denoise over, then the sequence lengths advance by one block.
#include "common.h"

namespace herald {
namespace {

// grid (block, Hkv, batch); one lane per 16-byte chunk of a row.
__global__ void append_kernel(const char *__restrict__ done_k, const char *__restrict__ done_v,
                              PoolView cache, const int32_t *__restrict__ seq_lens,
                              PoolView idle, const int32_t *__restrict__ k_next, int k_max,
                              int block, int Hkv, int row_bytes, int elt, int64_t cache_cap) {
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int c = threadIdx.x;
  if (c * 16 >= row_bytes) return;
  const int64_t S = seq_lens[b];
  if (S < 0 || S + block > cache_cap) return;  // lengths outside the cache: no write
  const int64_t src = (((int64_t)b * block + i) * Hkv + h) * row_bytes + c * 16;
  const uint4 kx = ldg16(done_k + src);
  const uint4 vx = ldg16(done_v + src);
  const int64_t dc = ((int64_t)b * cache.sb + (int64_t)h * cache.sh + (S + i) * cache.ss) * elt + c * 16;
  *reinterpret_cast<uint4 *>(cache.k + dc) = kx;
  *reinterpret_cast<uint4 *>(cache.v + dc) = vx;
  if (idle.k != nullptr) {
    const int kb = clamp_k(k_next[b], S, k_max);
    const int64_t di = ((int64_t)b * idle.sb + (int64_t)h * idle.sh + (int64_t)(kb + i) * idle.ss) * elt + c * 16;
    *reinterpret_cast<uint4 *>(idle.k + di) = kx;
    *reinterpret_cast<uint4 *>(idle.v + di) = vx;
  }
}

__global__ void bump_kernel(int batch, int block, int32_t *__restrict__ seq_lens,
                            int32_t *__restrict__ n_idle, const int32_t *__restrict__ k_next,
                            int k_max) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const int64_t S = seq_lens[b];
  if (n_idle != nullptr) n_idle[b] = clamp_k(k_next[b], S, k_max) + block;
  seq_lens[b] = (int32_t)(S + block);
}

}  // namespace

hipError_t launch_append(const herald_heads &hd, int batch, int block, const void *done_k,
                         const void *done_v, const PoolView &cache, const int32_t *seq_lens,
                         const PoolView *idle, const int32_t *k_next, int k_max,
                         int64_t cache_cap, hipStream_t stream) {
  const int elt = hd.dtype == HERALD_BF16 ? 2 : 4;
  const int rb = hd.head_dim * elt;
  PoolView none{nullptr, nullptr, 0, 0, 0};
  append_kernel<<<dim3(block, hd.num_kv_heads, batch), (rb + 15) / 16, 0, stream>>>(
      reinterpret_cast<const char *>(done_k), reinterpret_cast<const char *>(done_v), cache,
      seq_lens, idle ? *idle : none, k_next, k_max, block, hd.num_kv_heads, rb, elt, cache_cap);
  return hipGetLastError();
}

hipError_t launch_bump(int batch, int block, int32_t *seq_lens, int32_t *n_idle,
                       const int32_t *k_next, int k_max, hipStream_t stream) {
  bump_kernel<<<(batch + 255) / 256, 256, 0, stream>>>(batch, block, seq_lens, n_idle,
                                                        k_next, k_max);
  return hipGetLastError();
}

}  // namespace herald
