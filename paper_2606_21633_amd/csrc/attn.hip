// Block attention of the denoising phase (sec. II-A; sec. IV-B.2, where the
// main stream denoises block n from the active pool): every block query row
// attends to the context rows of its KV head (sparse pool or full cache)
// followed by the block's own B rows, with no mask.
//
// bf16 path, one workgroup = (key split, KV head x row block, sequence):
//   * the G*B query rows of a KV head are the MFMA "N" side: each wave owns
//     32 rows; its Q fragment stays in registers for the whole key loop;
//   * per 64-key tile, K is staged row-major and V transposed into LDS;
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 puts one query per lane
//     column, so the running max / sum of the online softmax need only one
//     cross-lane exchange (lane ^ 32);
//   * O^T = V^T P^T reuses the score registers directly as the B operand
//     (the V^T rows in LDS are stored in the matching key order), so P never
//     leaves registers and the O^T rescale is lane-local;
//   * with more than one key split, unnormalised partials (O, m, l) go to the
//     workspace and a combine kernel merges them.
// fp32 path: a plain VALU kernel (one wave per query row), exact expf.
#include <math.h>

#include "common.h"

namespace herald {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kKeyTile = 64;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// Byte offset of row `key` of (b, h) among context rows then block rows.
// Callers clamp key into [0, n_ctx + block).
__device__ __forceinline__ const char *row_ptr(const KvView &ctx, const char *ctxbase,
                                               const char *blk, int b, int h, int64_t key,
                                               int64_t n_ctx, int block, int Hkv, int D,
                                               int elt) {
  if (key < n_ctx) return ctxbase + kv_row(ctx, b, h, key) * elt;
  return blk + ((((int64_t)b * block + (key - n_ctx)) * Hkv + h) * D) * elt;
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};  // v_cvt_pk_bf16_f32, round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64, 2) void attn_bf16_kernel(
    const uint16_t *__restrict__ q, KvView ctx, const uint16_t *__restrict__ blk_k,
    const uint16_t *__restrict__ blk_v, uint16_t *__restrict__ out,
    float *__restrict__ part_o, float2 *__restrict__ part_ml, int block, int Hq, int Hkv,
    int G, int M, int n_mblk, int nsplit, int keys_per_split, float sl2) {
  constexpr int KT = kKeyTile;
  constexpr int KSTR = D * 2 + 16;   // LDS bytes per K row (padded)
  constexpr int VSTR = KT * 2 + 16;  // LDS bytes per V^T row (one d, padded)
  constexpr int NKS = D / 16;        // MFMA k-steps of K Q^T
  constexpr int NDT = D / 32;        // 32-wide d tiles of O^T
  constexpr int NTH = NW * 64;
  constexpr int CPR = D / 8;         // 16-byte chunks per row
  constexpr int KLD = KT * CPR / NTH;        // K chunks per thread per tile
  constexpr int VTASK = (KT / 4) * CPR;      // (4 keys, one chunk) V tasks per tile
  constexpr int VLD = (VTASK + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) char Ks[2][KT * KSTR];
  __shared__ __attribute__((aligned(16))) char Vt[2][D * VSTR];

  const int split = blockIdx.x;
  const int h = blockIdx.y / n_mblk, mblk = blockIdx.y % n_mblk;
  const int b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hh = lane >> 5, l32 = lane & 31;
  const int64_t n_ctx = kv_len(ctx, b);
  const int64_t n_keys = n_ctx + block;
  const int64_t k_begin = (int64_t)split * keys_per_split;
  const int64_t k_end = min(k_begin + (int64_t)keys_per_split, n_keys);

  const int r = (mblk * NW + wave) * 32 + l32;  // query row of this lane's column
  const bool rvalid = r < M;
  const int g = rvalid ? r / block : 0, i = rvalid ? r % block : 0;
  const int64_t qoff = ((((int64_t)b * block + i) * Hq + h * G + g) * D);
  bf16x8 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = rvalid ? as_bf16x8(ldg16(q + qoff + 8 * hh + 16 * ks))
                    : as_bf16x8(make_uint4(0u, 0u, 0u, 0u));

  f32x16 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[dt][j] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const char *ck = ctx.k, *cv = ctx.v;
  const char *bk = reinterpret_cast<const char *>(blk_k);
  const char *bv = reinterpret_cast<const char *>(blk_v);

  // ---- global -> registers for one tile (keys past the end re-read the last
  // valid row; their scores are masked) -------------------------------------
  uint4 kreg[KLD];
  uint4 vreg[VLD][4];
  auto fetch = [&](int64_t t0) {
#pragma unroll
    for (int u = 0; u < KLD; ++u) {
      const int x = tid + u * NTH;
      const int kk = x / CPR, c = x % CPR;
      const int64_t key = min(t0 + kk, k_end - 1);
      kreg[u] = ldg16(row_ptr(ctx, ck, bk, b, h, key, n_ctx, block, Hkv, D, 2) + c * 16);
    }
#pragma unroll
    for (int u = 0; u < VLD; ++u) {
      const int x = tid + u * NTH;
      if (VTASK % NTH == 0 || x < VTASK) {
        const int kg = x % (KT / 4), c = x / (KT / 4);
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int64_t key = min(t0 + kg * 4 + a, k_end - 1);
          vreg[u][a] = ldg16(row_ptr(ctx, cv, bv, b, h, key, n_ctx, block, Hkv, D, 2) + c * 16);
        }
      }
    }
  };
  // ---- registers -> LDS: K row-major; V transposed, where inside each group
  // of 16 keys key 8a + 4p + x sits at position 8p + 4a + x (the order in
  // which the score registers feed the P^T operand) -------------------------
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < KLD; ++u) {
      const int x = tid + u * NTH;
      const int kk = x / CPR, c = x % CPR;
      *reinterpret_cast<uint4 *>(Ks[buf] + kk * KSTR + c * 16) = kreg[u];
    }
#pragma unroll
    for (int u = 0; u < VLD; ++u) {
      const int x = tid + u * NTH;
      if (VTASK % NTH == 0 || x < VTASK) {
        const int kg = x % (KT / 4), c = x / (KT / 4);
        const int kk0 = kg * 4;
        const int pos0 = (kk0 & ~15) | (((kk0 >> 2) & 1) << 3) | (((kk0 >> 3) & 1) << 2);
        const uint32_t w0[4] = {vreg[u][0].x, vreg[u][0].y, vreg[u][0].z, vreg[u][0].w};
        const uint32_t w1[4] = {vreg[u][1].x, vreg[u][1].y, vreg[u][1].z, vreg[u][1].w};
        const uint32_t w2[4] = {vreg[u][2].x, vreg[u][2].y, vreg[u][2].z, vreg[u][2].w};
        const uint32_t w3[4] = {vreg[u][3].x, vreg[u][3].y, vreg[u][3].z, vreg[u][3].w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          // d = 8c + 2p (low halves) and 8c + 2p + 1 (high halves)
          uint2 lo, hi;
          lo.x = __builtin_amdgcn_perm(w1[p], w0[p], 0x05040100u);
          lo.y = __builtin_amdgcn_perm(w3[p], w2[p], 0x05040100u);
          hi.x = __builtin_amdgcn_perm(w1[p], w0[p], 0x07060302u);
          hi.y = __builtin_amdgcn_perm(w3[p], w2[p], 0x07060302u);
          *reinterpret_cast<uint2 *>(Vt[buf] + (8 * c + 2 * p) * VSTR + pos0 * 2) = lo;
          *reinterpret_cast<uint2 *>(Vt[buf] + (8 * c + 2 * p + 1) * VSTR + pos0 * 2) = hi;
        }
      }
    }
  };

  if (k_begin < k_end) {
    fetch(k_begin);
    stash(0);
  }
  __syncthreads();
  int cur = 0;
  for (int64_t t0 = k_begin; t0 < k_end; t0 += KT) {
    const bool more = t0 + KT < k_end;
    if (more) fetch(t0 + KT);  // in flight while this tile is computed

    // S^T (keys x queries) for the two 32-key halves of the tile
    f32x16 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int j = 0; j < 16; ++j) s[t][j] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4 *>(
            Ks[cur] + (32 * t + l32) * KSTR + (8 * hh + 16 * ks) * 2));
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[t], 0, 0, 0);
      }
    }
    // online softmax in the log2 domain; lane (l32, hh) holds keys
    // 32t + 8(j/4) + 4hh + j%4 of query column l32
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 16; ++j) s[t][j] *= sl2;
    if (t0 + KT > k_end) {  // last, partial tile
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int64_t key = t0 + 32 * t + 8 * (j >> 2) + 4 * hh + (j & 3);
          if (key >= k_end) s[t][j] = -INFINITY;
        }
    }
    float mx = s[0][0];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[t][j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = __builtin_amdgcn_exp2f(s[t][j] - m_new);
        s[t][j] = p;
        psum += p;
      }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    if (__ballot(alpha != 1.f)) {  // the running max moved for some row
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[dt][j] *= alpha;
    }

    // O^T += V^T P^T, four 16-key steps
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int t = ks >> 1, base = (ks & 1) * 8;
      uint4 pw;
      pw.x = pack2(s[t][base + 0], s[t][base + 1]);
      pw.y = pack2(s[t][base + 2], s[t][base + 3]);
      pw.z = pack2(s[t][base + 4], s[t][base + 5]);
      pw.w = pack2(s[t][base + 6], s[t][base + 7]);
      const bf16x8 pb = as_bf16x8(pw);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4 *>(
            Vt[cur] + (32 * dt + l32) * VSTR + (16 * ks + 8 * hh) * 2));
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[dt], 0, 0, 0);
      }
    }
    if (more) stash(cur ^ 1);
    __syncthreads();
    cur ^= 1;
  }

  if (!rvalid) return;
  // lane holds d = 32dt + 8(j/4) + 4hh + j%4 of query row r
  if (nsplit == 1) {
    const float inv = 1.f / l_run;
    uint16_t *orow = out + qoff;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        uint2 w;
        w.x = pack2(o[dt][4 * i4 + 0] * inv, o[dt][4 * i4 + 1] * inv);
        w.y = pack2(o[dt][4 * i4 + 2] * inv, o[dt][4 * i4 + 3] * inv);
        *reinterpret_cast<uint2 *>(orow + 32 * dt + 8 * i4 + 4 * hh) = w;
      }
  } else {
    const int64_t p = ((int64_t)b * Hkv + h) * nsplit + split;
    float *po = part_o + (p * M + r) * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
        *reinterpret_cast<float4 *>(po + 32 * dt + 8 * i4 + 4 * hh) =
            make_float4(o[dt][4 * i4 + 0], o[dt][4 * i4 + 1], o[dt][4 * i4 + 2],
                        o[dt][4 * i4 + 3]);
    if (hh == 0) part_ml[p * M + r] = make_float2(m_run, l_run);
  }
}

// Merge of split-KV partials (log2-domain statistics), 4 outputs per thread.
__global__ __launch_bounds__(256) void attn_combine_kernel(
    const float *__restrict__ part_o, const float2 *__restrict__ part_ml,
    uint16_t *__restrict__ out, int block, int Hq, int Hkv, int G, int M, int D,
    int nsplit) {
  const int h = blockIdx.y, b = blockIdx.z;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int r = idx / (D / 4), d0 = (idx % (D / 4)) * 4;
  if (r >= M) return;
  const int64_t p0 = ((int64_t)b * Hkv + h) * nsplit;
  float mx = -INFINITY;
  for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, part_ml[(p0 + s) * M + r].x);
  float den = 0.f, n0 = 0.f, n1 = 0.f, n2 = 0.f, n3 = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float2 ml = part_ml[(p0 + s) * M + r];
    if (ml.x == -INFINITY) continue;
    const float w = __builtin_amdgcn_exp2f(ml.x - mx);
    const float4 v = *reinterpret_cast<const float4 *>(part_o + ((p0 + s) * M + r) * D + d0);
    den += ml.y * w;
    n0 += v.x * w; n1 += v.y * w; n2 += v.z * w; n3 += v.w * w;
  }
  const float inv = 1.f / den;
  const int g = r / block, i = r % block;
  uint16_t *orow = out + (((int64_t)b * block + i) * Hq + h * G + g) * D + d0;
  uint2 w;
  w.x = pack2(n0 * inv, n1 * inv);
  w.y = pack2(n2 * inv, n3 * inv);
  *reinterpret_cast<uint2 *>(orow) = w;
}

// fp32 path: one wave per query row; lanes split the keys of a 64-key pass,
// then accumulate P V with the probabilities broadcast across the wave.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float *__restrict__ q, KvView ctx, const float *__restrict__ blk_k,
    const float *__restrict__ blk_v, float *__restrict__ out, int block, int Hq, int Hkv,
    int G, int M, float scale) {
  constexpr int ND = (D + 63) / 64;
  const int h = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= M) return;
  const int g = r / block, i = r % block;
  const int64_t qoff = (((int64_t)b * block + i) * Hq + h * G + g) * D;
  const int64_t n_ctx = kv_len(ctx, b);
  const int64_t n_keys = n_ctx + block;
  const char *ck = ctx.k, *cv = ctx.v;
  const char *bk = reinterpret_cast<const char *>(blk_k);
  const char *bv = reinterpret_cast<const char *>(blk_v);
  float m = -INFINITY, l = 0.f, o[ND];
#pragma unroll
  for (int u = 0; u < ND; ++u) o[u] = 0.f;
  for (int64_t j0 = 0; j0 < n_keys; j0 += 64) {
    const int64_t key = j0 + lane;
    float logit = -INFINITY;
    if (key < n_keys) {
      const float *kr = reinterpret_cast<const float *>(
          row_ptr(ctx, ck, bk, b, h, key, n_ctx, block, Hkv, D, 4));
      float acc = 0.f;
      for (int e = 0; e < D; ++e) acc = fmaf(q[qoff + e], kr[e], acc);
      logit = acc * scale;
    }
    float pm = logit;
    for (int off = 32; off >= 1; off >>= 1) pm = fmaxf(pm, __shfl_xor(pm, off, 64));
    const float m_new = fmaxf(m, pm);
    const float alpha = expf(m - m_new);
    const float p = expf(logit - m_new);
    float ps = p;
    for (int off = 32; off >= 1; off >>= 1) ps += __shfl_xor(ps, off, 64);
    l = l * alpha + ps;
    m = m_new;
#pragma unroll
    for (int u = 0; u < ND; ++u) o[u] *= alpha;
    const int nvalid = (int)min((int64_t)64, n_keys - j0);
    for (int jj = 0; jj < nvalid; ++jj) {
      const float pj = __shfl(p, jj, 64);
      const float *vr = reinterpret_cast<const float *>(
          row_ptr(ctx, cv, bv, b, h, j0 + jj, n_ctx, block, Hkv, D, 4));
#pragma unroll
      for (int u = 0; u < ND; ++u) {
        const int d = lane + 64 * u;
        if (d < D) o[u] = fmaf(pj, vr[d], o[u]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < ND; ++u) {
    const int d = lane + 64 * u;
    if (d < D) out[qoff + d] = o[u] / l;
  }
}

// Workgroups the split-KV plan aims for; read once per process.
int target_wgs() {
  static const int t = [] {
    const char *v = getenv("HERALD_ATTN_TARGET_WGS");
    const int x = v ? atoi(v) : 512;
    return x > 0 ? x : 512;
  }();
  return t;
}

}  // namespace

AttnPlan attn_plan(const herald_heads &hd, int batch, int block, int64_t max_ctx) {
  AttnPlan p{};
  const int G = hd.num_q_heads / hd.num_kv_heads;
  p.M = G * block;
  p.nsplit = 1;
  p.nsplit_cap = 1;
  p.keys_per_split = (int)(max_ctx + block);
  if (hd.dtype != HERALD_BF16) {
    p.nwaves = 4;
    p.n_mblk = (p.M + 3) / 4;
    return p;
  }
  p.nwaves = p.M > 64 ? 4 : (p.M > 32 ? 2 : 1);
  p.n_mblk = (p.M + 32 * p.nwaves - 1) / (32 * p.nwaves);
  const int64_t max_keys = max_ctx + block;
  const int64_t ntile = (max_keys + kKeyTile - 1) / kKeyTile;
  const int64_t base = (int64_t)batch * hd.num_kv_heads * p.n_mblk;
  int64_t want = (target_wgs() + base - 1) / base;
  if (want < 1) want = 1;
  const int64_t ns = want < ntile ? want : ntile;
  const int64_t tiles_per = (ntile + ns - 1) / ns;
  p.keys_per_split = (int)(tiles_per * kKeyTile);
  p.nsplit = (int)((max_keys + p.keys_per_split - 1) / p.keys_per_split);
  // nsplit <= min(want, ntile), which grows with the context: sizing the
  // partials by it covers every shorter context too
  p.nsplit_cap = (int)ns;
  if (p.nsplit_cap > 1) {
    const size_t parts = (size_t)batch * hd.num_kv_heads * p.nsplit_cap * p.M;
    p.part_o_bytes = parts * hd.head_dim * sizeof(float);
    p.part_ml_bytes = parts * sizeof(float2);
  }
  return p;
}

hipError_t launch_block_attn(const herald_heads &hd, int batch, int block, const void *q,
                             const KvView &ctx, int64_t max_ctx, const void *blk_k,
                             const void *blk_v, void *out, void *ws, hipStream_t stream) {
  const AttnPlan p = attn_plan(hd, batch, block, max_ctx);
  const int G = hd.num_q_heads / hd.num_kv_heads;
  const int Hq = hd.num_q_heads, Hkv = hd.num_kv_heads, D = hd.head_dim;
  if (hd.dtype != HERALD_BF16) {
    const dim3 grid(p.n_mblk, Hkv, batch);
    const float scale = (float)(1.0 / sqrt((double)D));
    if (D == 64)
      attn_f32_kernel<64><<<grid, 256, 0, stream>>>(
          (const float *)q, ctx, (const float *)blk_k, (const float *)blk_v, (float *)out,
          block, Hq, Hkv, G, p.M, scale);
    else if (D == 128)
      attn_f32_kernel<128><<<grid, 256, 0, stream>>>(
          (const float *)q, ctx, (const float *)blk_k, (const float *)blk_v, (float *)out,
          block, Hq, Hkv, G, p.M, scale);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  char *w = reinterpret_cast<char *>(ws);
  float *part_o = reinterpret_cast<float *>(w);
  float2 *part_ml = reinterpret_cast<float2 *>(w + ((p.part_o_bytes + 255) & ~(size_t)255));
  const float sl2 = (float)(1.0 / sqrt((double)D)) * kLog2e;
  const dim3 grid(p.nsplit, Hkv * p.n_mblk, batch);
  const uint16_t *qq = (const uint16_t *)q;
  const uint16_t *bk = (const uint16_t *)blk_k, *bv = (const uint16_t *)blk_v;
  uint16_t *oo = (uint16_t *)out;
#define HERALD_ATTN(D_, NW_)                                                            \
  if (D == D_ && p.nwaves == NW_)                                                       \
    attn_bf16_kernel<D_, NW_><<<grid, NW_ * 64, 0, stream>>>(                           \
        qq, ctx, bk, bv, oo, part_o, part_ml, block, Hq, Hkv, G, p.M, p.n_mblk,        \
        p.nsplit, p.keys_per_split, sl2);
  HERALD_ATTN(64, 1) else HERALD_ATTN(64, 2) else HERALD_ATTN(64, 4)
  else HERALD_ATTN(128, 1) else HERALD_ATTN(128, 2) else HERALD_ATTN(128, 4)
  else return hipErrorInvalidValue;
#undef HERALD_ATTN
  if (p.nsplit > 1) {
    const dim3 cg((p.M * (D / 4) + 255) / 256, Hkv, batch);
    attn_combine_kernel<<<cg, 256, 0, stream>>>(part_o, part_ml, oo, block, Hq, Hkv, G,
                                                p.M, D, p.nsplit);
  }
  return hipGetLastError();
}

}  // namespace herald
