// Gather of the selected K/V rows into a sparse pool (sec. IV-B.3 of the
// paper: the selected entries are copied into a contiguous buffer that the
// denoising phase reads). On one GPU this is an HBM-to-HBM copy of random
// cache rows into contiguous pool rows; it is bandwidth-bound.
//
// One workgroup copies kRowsPerWg pool rows of one (KV head, sequence); each
// row is moved by 16-byte lanes (a 256-byte bf16 d=128 row is 16 lanes), K and
// V both, so every load and store is a full 128-bit access.
#include "common.h"

namespace herald {
namespace {

constexpr int kGatherThreads = 256;
constexpr int kRowsPerWg = 64;

template <int RB, bool PAGED>
__global__ __launch_bounds__(kGatherThreads) void gather_kernel(
    KvView kv, const int32_t *__restrict__ idx, const int32_t *__restrict__ kps,
    int k_max, PoolView dst, int dst_row0, int Hkv, int elt) {
  constexpr int LPR = RB / 16;                   // lanes per row
  constexpr int RPI = kGatherThreads / LPR;      // rows per iteration
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t S = kv_len(kv, b);
  const int k = clamp_k(kps[b], S, k_max);
  const int j0 = blockIdx.x * kRowsPerWg;
  if (j0 >= k) return;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int lr = threadIdx.x / LPR, lc = threadIdx.x % LPR;
  constexpr int NIT = kRowsPerWg / RPI;
  // every index, then every row load, then every store: NIT rows of K and V
  // in flight per thread (a row whose index is out of range, or past k, is
  // skipped; herald_select produces none of the former)
  int64_t s[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = j0 + it * RPI + lr;
    const int32_t x = idx[bh * k_max + min(j, k - 1)];  // (row k - 1 re-read, unused)
    s[it] = j < k ? (int64_t)x : -1;
  }
  // a skipped row loads row 0 of the sequence (in bounds) and stores nothing
  uint4 kx[NIT], vx[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int64_t row = s[it] >= 0 && s[it] < S ? s[it] : 0;
    const int64_t src =
        (PAGED ? kv_row(kv, b, h, row) : (int64_t)b * kv.sb + (int64_t)h * kv.sh + row * kv.ss) *
            elt + lc * 16;
    kx[it] = ldg16(kv.k + src);
    vx[it] = ldg16(kv.v + src);
  }
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    if (s[it] < 0 || s[it] >= S) continue;
    const int j = j0 + it * RPI + lr;
    const int64_t d = ((int64_t)b * dst.sb + (int64_t)h * dst.sh +
                       (int64_t)(dst_row0 + j) * dst.ss) * elt + lc * 16;
    *reinterpret_cast<uint4 *>(dst.k + d) = kx[it];
    *reinterpret_cast<uint4 *>(dst.v + d) = vx[it];
  }
}

}  // namespace

hipError_t launch_gather(const herald_heads &hd, int batch, const KvView &kv,
                         const int32_t *idx, const int32_t *k_per_seq, int k_max,
                         const PoolView &dst, int dst_row0, hipStream_t stream) {
  const int elt = hd.dtype == HERALD_BF16 ? 2 : 4;
  const int rb = hd.head_dim * elt;
  const dim3 grid((k_max + kRowsPerWg - 1) / kRowsPerWg, hd.num_kv_heads, batch);
  const bool paged = kv.pt != nullptr;
#define HERALD_GATHER(RB_)                                                                    \
  case RB_:                                                                                  \
    if (paged)                                                                               \
      gather_kernel<RB_, true><<<grid, kGatherThreads, 0, stream>>>(                          \
          kv, idx, k_per_seq, k_max, dst, dst_row0, hd.num_kv_heads, elt);                   \
    else                                                                                     \
      gather_kernel<RB_, false><<<grid, kGatherThreads, 0, stream>>>(                         \
          kv, idx, k_per_seq, k_max, dst, dst_row0, hd.num_kv_heads, elt);                   \
    break;
  switch (rb) {
    HERALD_GATHER(128)
    HERALD_GATHER(256)
    HERALD_GATHER(512)
    default: return hipErrorInvalidValue;
  }
#undef HERALD_GATHER
  return hipGetLastError();
}

}  // namespace herald
