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

typedef __attribute__((ext_vector_type(4))) float f32x4;

// Max over the four lanes l, l^16, l^32, l^48 that hold the keys of one
// query column, with the gfx950 half-row swaps (no LDS traffic).
__device__ __forceinline__ float max4q(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  return fmaxf(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

// One workgroup: P pipelines of NW waves. Each wave owns 16 query rows (the
// MFMA N side of v_mfma_f32_16x16x32_bf16), each pipeline takes every P-th
// key tile of the workgroup's key range, and the pipelines are merged in LDS
// at the end. KT keys per tile: K row-major and V transposed in LDS, double
// buffered per pipeline, one barrier per tile.
template <int D, int NW, int P, int KT, bool PAGED>
__global__ __launch_bounds__(NW * P * 64, 1) void attn_bf16_kernel(
    const uint16_t *__restrict__ q, KvView ctx, const uint16_t *__restrict__ blk_k,
    const uint16_t *__restrict__ blk_v, uint16_t *__restrict__ out,
    float *__restrict__ part_o, float2 *__restrict__ part_ml, int block, int Hq, int Hkv,
    int G, int M, int n_mblk, int nsplit, int keys_per_split, float sl2) {
  constexpr int KSTR = D * 2 + 16;   // LDS bytes per K row (padded)
  constexpr int VSTR = KT * 2 + 16;  // LDS bytes per V^T row (one d, padded)
  constexpr int NKS = D / 32;        // k-steps of K Q^T (32 d each)
  constexpr int NKB = KT / 16;       // 16-key blocks per tile
  constexpr int NDB = D / 16;        // 16-d blocks of O^T
  constexpr int NPS = KT / 32;       // k-steps of V^T P^T (32 keys each)
  constexpr int NTH = NW * 64;       // threads per pipeline
  constexpr int CPR = D / 8;         // 16-byte chunks per row
  constexpr int KLD = KT * CPR / NTH;
  // V is staged as tasks of TK consecutive keys x one 16-byte chunk; two-key
  // tasks when four-key ones would leave threads of the pipeline idle
  constexpr int TK = (KT / 4) * CPR >= NTH ? 4 : 2;
  constexpr int VTASK = (KT / TK) * CPR;
  constexpr int VLD = (VTASK + NTH - 1) / NTH;
  constexpr int KBYTES = KT * KSTR, VBYTES = D * VSTR;
  constexpr int STAGE = KBYTES + VBYTES;     // one buffer of one pipeline
  static_assert(KLD * NTH == KT * CPR, "K tile must split evenly over a pipeline");
  extern __shared__ __attribute__((aligned(16))) char smem[];

  // Workgroups are dealt round-robin to the 8 XCDs by linear id. When the row
  // blocks of one KV head split its query rows, place them on the same XCD
  // (ids id and id + 8, ...) so that their shared K/V tiles hit its L2.
  int split = blockIdx.x, b = blockIdx.z, h, mblk;
  {
    const int y = blockIdx.y;
    h = y / n_mblk;
    mblk = y % n_mblk;
    const int pairs = gridDim.y / n_mblk * gridDim.z;   // (b, h) pairs
    if (gridDim.x == 1 && n_mblk > 1 && pairs % 8 == 0) {
      const int id = y + gridDim.y * blockIdx.z;
      const int slot = id / 8;
      mblk = slot % n_mblk;
      const int pair = (slot / n_mblk) * 8 + id % 8;
      const int hk = gridDim.y / n_mblk;
      b = pair / hk;
      h = pair % hk;
    }
  }
  const int pipe = threadIdx.x / NTH;
  const int tid = threadIdx.x % NTH, wave = tid >> 6, lane = tid & 63;
  const int q4 = lane >> 4, l16 = lane & 15;
  const int64_t n_ctx = kv_len(ctx, b);
  const int64_t n_keys = n_ctx + block;
  const int64_t k_begin = (int64_t)split * keys_per_split;
  const int64_t k_end = min(k_begin + (int64_t)keys_per_split, n_keys);
  char *my = smem + pipe * 2 * STAGE;

  const int r = (mblk * NW + wave) * 16 + l16;  // query row of this lane's column
  const bool rvalid = r < M;
  const int g = rvalid ? r / block : 0, i = rvalid ? r % block : 0;
  const int64_t qoff = ((((int64_t)b * block + i) * Hq + h * G + g) * D);
  bf16x8 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = rvalid ? as_bf16x8(ldg16(q + qoff + 32 * ks + 8 * q4))
                    : as_bf16x8(make_uint4(0u, 0u, 0u, 0u));
  // o[NDB] accumulates the softmax denominator (a block of ones times P^T)
  f32x4 o[NDB + 1];
#pragma unroll
  for (int db = 0; db <= NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // reference max of raw scores
  const bf16x8 ones = as_bf16x8(make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u));

  // Row `key` of (b, h): the first n_ctx keys are context rows, the next
  // `block` keys the block's own rows. Contiguous contexts and the block rows
  // are both linear in the key, so the address is a select, not a branch.
  const char *bk = reinterpret_cast<const char *>(blk_k) +
                   (((int64_t)b * block * Hkv + h) * D - n_ctx * Hkv * D) * 2;
  const char *bv = reinterpret_cast<const char *>(blk_v) +
                   (((int64_t)b * block * Hkv + h) * D - n_ctx * Hkv * D) * 2;
  const int64_t brs = (int64_t)Hkv * D * 2;   // block row stride (bytes)
  const int64_t crs = ctx.ss * 2;             // context row stride (bytes)
  const char *ckb = ctx.k + ((int64_t)b * ctx.sb + (int64_t)h * ctx.sh) * 2;
  const char *cvb = ctx.v + ((int64_t)b * ctx.sb + (int64_t)h * ctx.sh) * 2;
  auto kaddr = [&](const char *cbase, const char *bbase, bool v, int64_t key) -> const char * {
    key = min(key, k_end - 1);
    if (PAGED && key < n_ctx) return (v ? ctx.v : ctx.k) + kv_row(ctx, b, h, key) * 2;
    return key < n_ctx ? cbase + key * crs : bbase + key * brs;
  };

  uint4 kreg[KLD];
  uint4 vreg[VLD][TK];
  // per-thread byte offsets inside a tile of contiguous context rows
  uint32_t koff[KLD], voff[VLD];
#pragma unroll
  for (int u = 0; u < KLD; ++u) {
    const int x = tid + u * NTH;
    koff[u] = (uint32_t)((x / CPR) * crs + (x % CPR) * 16);
  }
#pragma unroll
  for (int u = 0; u < VLD; ++u) {
    const int x = tid + u * NTH;
    voff[u] = (uint32_t)(((x % (KT / TK)) * TK) * crs + (x / (KT / TK)) * 16);
  }
  // global -> registers for the tile at t0. A tile wholly inside a
  // contiguous context is a uniform base plus the offsets above; otherwise
  // keys past the end re-read the last valid row (their scores are masked).
  auto fetch = [&](int64_t t0) {
    if (!PAGED && t0 + KT <= n_ctx && t0 + KT <= k_end) {
      const char *kt = ckb + t0 * crs, *vt = cvb + t0 * crs;
#pragma unroll
      for (int u = 0; u < KLD; ++u) kreg[u] = ldg16(kt + koff[u]);
#pragma unroll
      for (int u = 0; u < VLD; ++u) {
        const int x = tid + u * NTH;
        if (VTASK % NTH == 0 || x < VTASK) {
#pragma unroll
          for (int a = 0; a < TK; ++a) vreg[u][a] = ldg16(vt + voff[u] + a * crs);
        }
      }
      return;
    }
    asm volatile("");  // keep this path a branch
#pragma unroll
    for (int u = 0; u < KLD; ++u) {
      const int x = tid + u * NTH;
      const int kk = x / CPR, c = x % CPR;
      kreg[u] = ldg16(kaddr(ckb, bk, false, t0 + kk) + c * 16);
    }
#pragma unroll
    for (int u = 0; u < VLD; ++u) {
      const int x = tid + u * NTH;
      if (VTASK % NTH == 0 || x < VTASK) {
        const int kg = x % (KT / TK), c = x / (KT / TK);
#pragma unroll
        for (int a = 0; a < TK; ++a)
          vreg[u][a] = ldg16(kaddr(cvb, bv, true, t0 + kg * TK + a) + c * 16);
      }
    }
  };
  // registers -> LDS: K row-major; V transposed. Inside each group of 32 keys
  // key 16a + 4q + x sits at position 8q + 4a + x: the order in which a lane's
  // score registers feed the P^T operand of one 32-key k-step.
  auto stash = [&](int buf) {
    char *Ks = my + buf * STAGE, *Vt = Ks + KBYTES;
#pragma unroll
    for (int u = 0; u < KLD; ++u) {
      const int x = tid + u * NTH;
      const int kk = x / CPR, c = x % CPR;
      *reinterpret_cast<uint4 *>(Ks + kk * KSTR + c * 16) = kreg[u];
    }
#pragma unroll
    for (int u = 0; u < VLD; ++u) {
      const int x = tid + u * NTH;
      if (VTASK % NTH == 0 || x < VTASK) {
        const int kg = x % (KT / TK), c = x / (KT / TK);
        const int kk0 = kg * TK;
        const int pos0 = (kk0 & ~31) | (((kk0 >> 2) & 3) << 3) | (((kk0 >> 4) & 1) << 2) |
                         (kk0 & 3);
        const uint32_t w0[4] = {vreg[u][0].x, vreg[u][0].y, vreg[u][0].z, vreg[u][0].w};
        const uint32_t w1[4] = {vreg[u][1].x, vreg[u][1].y, vreg[u][1].z, vreg[u][1].w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          // d = 8c + 2p (low halves) and 8c + 2p + 1 (high halves)
          const uint32_t lo01 = __builtin_amdgcn_perm(w1[p], w0[p], 0x05040100u);
          const uint32_t hi01 = __builtin_amdgcn_perm(w1[p], w0[p], 0x07060302u);
          char *dlo = Vt + (8 * c + 2 * p) * VSTR + pos0 * 2;
          char *dhi = Vt + (8 * c + 2 * p + 1) * VSTR + pos0 * 2;
          if (TK == 4) {
            const uint32_t w2 = (&vreg[u][TK > 2 ? 2 : 0].x)[p];
            const uint32_t w3 = (&vreg[u][TK > 2 ? 3 : 0].x)[p];
            *reinterpret_cast<uint2 *>(dlo) =
                make_uint2(lo01, __builtin_amdgcn_perm(w3, w2, 0x05040100u));
            *reinterpret_cast<uint2 *>(dhi) =
                make_uint2(hi01, __builtin_amdgcn_perm(w3, w2, 0x07060302u));
          } else {
            *reinterpret_cast<uint32_t *>(dlo) = lo01;
            *reinterpret_cast<uint32_t *>(dhi) = hi01;
          }
        }
      }
    }
  };

  // pipeline `pipe` takes tiles pipe, pipe + P, ... of [k_begin, k_end)
  const int64_t ntile = (k_end - k_begin + KT - 1) / KT;
  const int64_t iters = (ntile + P - 1) / P;
  auto tile_start = [&](int64_t it) { return k_begin + (P * it + pipe) * KT; };
  if (iters > 0 && tile_start(0) < k_end) {
    fetch(tile_start(0));
    stash(0);
  }
  // The Q fragments stay in registers for the whole key loop: wait for them
  // here (their loads overlapped the first tile's) so that no wait on them
  // is left for the loop body.
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) asm volatile("" ::"v"(qf[ks]));
  __syncthreads();
  int cur = 0;
  for (int64_t it = 0; it < iters; ++it) {
    const int64_t t0 = tile_start(it);
    const bool active = t0 < k_end;                 // uniform per pipeline
    const bool more = tile_start(it + 1) < k_end;
    if (more) fetch(tile_start(it + 1));            // in flight during this tile
    if (active) {
      const char *Ks = my + cur * STAGE, *Vt = Ks + KBYTES;
      // S^T (keys x queries), one 16-key block at a time; lane (l16, q4)
      // holds keys 16kb + 4q4 + j of query column l16
      f32x4 s[NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        bf16x8 a[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
          a[ks] = as_bf16x8(*reinterpret_cast<const uint4 *>(
              Ks + (16 * kb + l16) * KSTR + (32 * ks + 8 * q4) * 2));
        s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
          s[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], qf[ks], s[kb], 0, 0, 0);
      }
      // online softmax on raw scores; the scale and log2(e) enter through
      // one FMA in the exp2 argument
      if (t0 + KT > k_end) {  // last, partial tile
        asm volatile("");     // keep this a branch: full tiles skip it
        const int lim = (int)(k_end - t0);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (16 * kb + 4 * q4 + j >= lim) s[kb][j] = -INFINITY;
      }
      float mx = s[0][0];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) mx = fmaxf(mx, s[kb][j]);
      mx = max4q(mx);
      // Lazy rescaling: the reference max m_run moves only when a row's max
      // exceeds it by more than 2^8 in probability (or on the first tile);
      // otherwise probabilities up to 256 are accumulated against the old
      // reference, which bf16 P and fp32 O hold exactly as well.
      if (__ballot((mx - m_run) * sl2 > 8.f)) {
        const float m_new = fmaxf(m_run, mx);
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * sl2);
#pragma unroll
        for (int db = 0; db < NDB + 1; ++db) o[db] *= alpha;
        m_run = m_new;
      }
      const float nb = -m_run * sl2;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) s[kb][j] = __builtin_amdgcn_exp2f(fmaf(s[kb][j], sl2, nb));
      // O^T += V^T P^T, one 32-key k-step at a time; the extra block of
      // ones gives the softmax denominator from the same bf16 P
#pragma unroll
      for (int ps = 0; ps < NPS; ++ps) {
        uint4 pw;
        pw.x = pack2(s[2 * ps][0], s[2 * ps][1]);
        pw.y = pack2(s[2 * ps][2], s[2 * ps][3]);
        pw.z = pack2(s[2 * ps + 1][0], s[2 * ps + 1][1]);
        pw.w = pack2(s[2 * ps + 1][2], s[2 * ps + 1][3]);
        const bf16x8 pb = as_bf16x8(pw);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 av = as_bf16x8(*reinterpret_cast<const uint4 *>(
              Vt + (16 * db + l16) * VSTR + (32 * ps + 8 * q4) * 2));
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb, o[db], 0, 0, 0);
        }
        o[NDB] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb, o[NDB], 0, 0, 0);
      }
    }
    if (more) stash(cur ^ 1);
    __syncthreads();
    cur ^= 1;
  }

  // merge pipelines 1..P-1 into pipeline 0 through LDS (same rows and lanes)
  if (P > 1) {
    constexpr int SLOT = (NDB + 1) * 4 + 1;
    float *xs = reinterpret_cast<float *>(smem);
    if (pipe > 0) {
      float *x = xs + ((size_t)(pipe - 1) * NTH + tid) * SLOT;
#pragma unroll
      for (int db = 0; db <= NDB; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) x[db * 4 + j] = o[db][j];
      x[(NDB + 1) * 4] = m_run;
    }
    __syncthreads();
    if (pipe > 0 || !rvalid) return;
#pragma unroll 1
    for (int pp = 1; pp < P; ++pp) {
      const float *x = xs + ((size_t)(pp - 1) * NTH + tid) * SLOT;
      const float m1 = x[(NDB + 1) * 4];
      const float mm = fmaxf(m_run, m1);
      const float a0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_run - mm) * sl2);
      const float a1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m1 - mm) * sl2);
#pragma unroll
      for (int db = 0; db <= NDB; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[db][j] = o[db][j] * a0 + x[db * 4 + j] * a1;
      m_run = mm;
    }
  } else if (!rvalid) {
    return;
  }
  const float l_run = o[NDB][0];
  // lane holds d = 16db + 4q4 + j of query row r
  if (nsplit == 1) {
    const float inv = 1.f / l_run;
    uint16_t *orow = out + qoff;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      uint2 w;
      w.x = pack2(o[db][0] * inv, o[db][1] * inv);
      w.y = pack2(o[db][2] * inv, o[db][3] * inv);
      *reinterpret_cast<uint2 *>(orow + 16 * db + 4 * q4) = w;
    }
  } else {
    const int64_t pidx = ((int64_t)b * Hkv + h) * nsplit + split;
    float *po = part_o + (pidx * M + r) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      *reinterpret_cast<float4 *>(po + 16 * db + 4 * q4) =
          make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
    if (q4 == 0) part_ml[pidx * M + r] = make_float2(m_run * sl2, l_run);
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
  // part_ml holds (max * scale * log2(e), sum) per row and split
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

// Query rows per workgroup (128 or 64); read once per process.
int max_rows_per_wg() {
  static const int r = [] {
    const char *v = getenv("HERALD_ATTN_ROWS");
    return (v && atoi(v) == 128) ? 128 : 64;
  }();
  return r;
}

// Workgroups the split-KV plan aims for; read once per process.
int target_wgs() {
  static const int t = [] {
    const char *v = getenv("HERALD_ATTN_TARGET_WGS");
    const int x = v ? atoi(v) : 256;
    return x > 0 ? x : 256;
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
  // waves of 16 rows; 128-row blocks run 2 pipelines of 64-key tiles, smaller
  // blocks 4 pipelines of 32-key tiles (both fill one CU's LDS)
  const int rows = max_rows_per_wg();
  p.nwaves = (p.M > 64 && rows >= 128) ? 8 : (p.M > 32 ? 4 : (p.M > 16 ? 2 : 1));
  p.pipes = p.nwaves == 8 ? 2 : 4;
  p.key_tile = p.nwaves == 8 ? 64 : 32;
  p.n_mblk = (p.M + 16 * p.nwaves - 1) / (16 * p.nwaves);
  const int64_t max_keys = max_ctx + block;
  const int64_t ntile = (max_keys + p.key_tile - 1) / p.key_tile;
  const int64_t base = (int64_t)batch * hd.num_kv_heads * p.n_mblk;
  // one workgroup per CU; every split gets at least one tile per pipeline
  int64_t want = (target_wgs() + base - 1) / base;
  if (want < 1) want = 1;
  const int64_t most = (ntile + p.pipes - 1) / p.pipes;
  const int64_t ns = want < most ? want : most;
  const int64_t tiles_per = (ntile + ns - 1) / ns;
  p.keys_per_split = (int)(tiles_per * p.key_tile);
  p.nsplit = (int)((max_keys + p.keys_per_split - 1) / p.keys_per_split);
  // nsplit <= min(want, ceil(ntile / pipes)), which grows with the context:
  // sizing the partials by it covers every shorter context too
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
  const bool paged = ctx.pt != nullptr;
#define HERALD_ATTN(D_, NW_, P_, KT_, PG_)                                               \
  if (D == D_ && p.nwaves == NW_ && paged == PG_) {                                      \
    auto kfn = attn_bf16_kernel<D_, NW_, P_, KT_, PG_>;                                  \
    constexpr int kSmem = 2 * P_ * (KT_ * (D_ * 2 + 16) + D_ * (KT_ * 2 + 16));          \
    static const hipError_t attr_err = hipFuncSetAttribute(                               \
        reinterpret_cast<const void *>(kfn), hipFuncAttributeMaxDynamicSharedMemorySize,  \
        kSmem);                                                                          \
    if (attr_err != hipSuccess) return attr_err;                                         \
    kfn<<<grid, NW_ * P_ * 64, kSmem, stream>>>(qq, ctx, bk, bv, oo, part_o, part_ml,     \
                                                block, Hq, Hkv, G, p.M, p.n_mblk,        \
                                                p.nsplit, p.keys_per_split, sl2);        \
  } else
  HERALD_ATTN(64, 8, 2, 64, false) HERALD_ATTN(64, 4, 4, 32, false)
  HERALD_ATTN(64, 2, 4, 32, false) HERALD_ATTN(64, 1, 4, 32, false)
  HERALD_ATTN(128, 8, 2, 64, false) HERALD_ATTN(128, 4, 4, 32, false)
  HERALD_ATTN(128, 2, 4, 32, false) HERALD_ATTN(128, 1, 4, 32, false)
  HERALD_ATTN(64, 8, 2, 64, true) HERALD_ATTN(64, 4, 4, 32, true)
  HERALD_ATTN(64, 2, 4, 32, true) HERALD_ATTN(64, 1, 4, 32, true)
  HERALD_ATTN(128, 8, 2, 64, true) HERALD_ATTN(128, 4, 4, 32, true)
  HERALD_ATTN(128, 2, 4, 32, true) HERALD_ATTN(128, 1, 4, 32, true)
  return hipErrorInvalidValue;
#undef HERALD_ATTN
  if (p.nsplit > 1) {
    const dim3 cg((p.M * (D / 4) + 255) / 256, Hkv, batch);
    attn_combine_kernel<<<cg, 256, 0, stream>>>(part_o, part_ml, oo, block, Hq, Hkv, G,
                                                p.M, D, p.nsplit);
  }
  return hipGetLastError();
}

}  // namespace herald
