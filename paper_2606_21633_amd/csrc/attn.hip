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

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// Byte offset of row `key` of (b, h) among context rows (of context sequence
// bc) then block rows. Callers clamp key into [0, n_ctx + block).
__device__ __forceinline__ const char *row_ptr(const KvView &ctx, const char *ctxbase,
                                               const char *blk, int bc, int b, int h,
                                               int64_t key, int64_t n_ctx, int block, int Hkv,
                                               int D, int elt) {
  if (key < n_ctx) return ctxbase + kv_row(ctx, bc, h, key) * elt;
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

typedef short __attribute__((ext_vector_type(4))) s16x4;
// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives element
// i % 4 of the 8 bytes addressed by lanes 4s + i / 4, for s = 0..3.
__device__ __forceinline__ uint2 lds_tr16(const char *p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4 *)(const __attribute__((address_space(3))) char *)p);
  return __builtin_bit_cast(uint2, v);
}
// Workgroup barrier that leaves global loads in flight (the fence of
// __syncthreads would wait for the register prefetch too); LDS writes are
// complete before it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Most query groups that attn_bf16_kernel orders by context length.
constexpr int kOrderMax = 256;

// LDS bytes of attn_bf16_kernel: the K/V ring (P pipelines x 2 stages of a
// 32-key K and V tile), or the pipeline merge area (the O blocks each wave
// hands to other pipelines and its (max, sum) per lane) if that is larger.
template <int D, int RW, int NWP, int P>
constexpr int attn_smem_bytes() {
  constexpr int ring = P * 2 * 2 * 32 * (2 * D);
  constexpr int merge =
      P > 1 ? P * NWP * (RW / 16) * 64 * ((D / 16 - D / 16 / P) * 16 + 8) : 0;
  static_assert(merge <= 160 * 1024, "merge area exceeds the LDS of a CU");
  return ring > merge ? ring : merge;
}

// One workgroup = ROWS = NWP * RW query rows of one KV head over one key
// split, as P pipelines of NWP waves. Pipeline p takes key tiles p, p + P, ...
// (KT = 32 keys each) and the pipelines are merged in LDS at the end. Each
// wave owns RW query rows: RW / 16 column blocks of v_mfma_f32_16x16x32_bf16
// that share every K and V operand the wave reads from LDS.
//
// Tiles go global -> registers -> LDS. Two register sets per thread hold the
// next two tiles of its pipeline while the current one is consumed from LDS
// (two LDS stages per pipeline), so every load has about two rounds to land.
// In LDS both K and V are row-major (2*D bytes per key) with the 16-byte
// chunks of row r XOR-swizzled: K by fK(r) so that the ds_read_b128 of 16
// rows in a quarter wave hit distinct banks, V by fV(r) so that the
// transposed ds_read_b64_tr_b16 (8 rows x 32 bytes per half wave) do.
template <int D, int RW, int NWP, int P, bool PAGED>
__global__ __launch_bounds__(NWP * P * 64, 1) void attn_bf16_kernel(
    const uint16_t *__restrict__ q, KvView ctx, const uint16_t *__restrict__ blk_k,
    const uint16_t *__restrict__ blk_v, uint16_t *__restrict__ out,
    float *__restrict__ part_o, float2 *__restrict__ part_ml, int block, int Hq, int Hkv,
    int G, int M, int n_mblk, int nsplit, int keys_per_split, float sl2, int groups,
    int order) {
  constexpr int KT = 32;             // keys per tile
  constexpr int CB = RW / 16;        // column blocks (16 query rows) per wave
  constexpr int NKS = D / 32;        // k-steps of K Q^T
  constexpr int NDB = D / 16;        // 16-d blocks of O^T
  constexpr int ROWB = 2 * D;        // bytes per K or V row
  constexpr int CPR = D / 8;         // 16-byte chunks per row
  constexpr int RSH = D == 64 ? 1 : 0;  // log2(rows per 256 bytes)
  constexpr int KB = KT * ROWB;      // bytes of one K (or V) tile
  constexpr int STAGE = 2 * KB;
  constexpr int NTH = NWP * 64;      // threads per pipeline
  constexpr int LPT = KT * CPR / NTH;  // 16-byte chunks per thread per K (or V) tile
  static_assert(LPT * NTH == KT * CPR, "tile must split evenly over a pipeline");
  extern __shared__ __attribute__((aligned(16))) char smem[];

  // Workgroups are dealt round-robin to the 8 XCDs by linear id. When the row
  // blocks of one KV head split its query rows, place them on the same XCD
  // (ids id and id + 8, ...) so that their shared K/V tiles hit its L2.
  // The grid is 1-D over (group, row block), a group being one (sequence, KV
  // head, key split). Workgroups are dealt round-robin to the 8 XCDs by id;
  // the row blocks of one group get ids id, id + 8, ... so that they run on
  // one XCD at the same time and share its L2 for their common K/V tiles.
  const int n_groups = gridDim.x / n_mblk;
  int grp, mblk;
  {
    const int id = blockIdx.x;
    if (n_mblk > 1 && n_groups % 8 == 0) {
      const int slot = id >> 3;
      mblk = slot % n_mblk;
      grp = (slot / n_mblk) * 8 + (id & 7);
    } else {
      mblk = id % n_mblk;
      grp = id / n_mblk;
    }
  }
  const int split = grp % nsplit;
  const int h = (grp / nsplit) % Hkv;
  int b = grp / nsplit / Hkv;
  if (order) {
    // More workgroups than CUs: the later ones start as earlier ones finish,
    // so b is taken as a rank and the query groups run longest context first
    // (ties to the lower index), leaving the short ones for the end of the
    // grid. Every thread takes part; the ranks are a permutation, so exactly
    // one query group matches.
    // (lengths padded with -1 to a multiple of 16, which rank below every
    // length, so the rank loop reads 16 at a time without a bound check)
    __shared__ __attribute__((aligned(16))) int lens_s[kOrderMax];
    __shared__ int pick_s;
    const int nb = gridDim.x / (n_mblk * nsplit * Hkv);
    const int nb16 = (nb + 15) & ~15;
    for (int j = threadIdx.x; j < nb16; j += blockDim.x)
      lens_s[j] = j < nb ? (int)kv_len(ctx, j / groups) : -1;
    __syncthreads();
    for (int j = threadIdx.x; j < nb; j += blockDim.x) {
      const int lj = lens_s[j];
      int rank = 0;
      for (int i0 = 0; i0 < nb16; i0 += 16) {
        int4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const int4 *>(lens_s + i0 + 4 * u);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = i0 + 4 * u;
          rank += (v[u].x > lj) | ((v[u].x == lj) & (i < j));
          rank += (v[u].y > lj) | ((v[u].y == lj) & (i + 1 < j));
          rank += (v[u].z > lj) | ((v[u].z == lj) & (i + 2 < j));
          rank += (v[u].w > lj) | ((v[u].w == lj) & (i + 3 < j));
        }
      }
      if (rank == b) pick_s = j;
    }
    __syncthreads();
    b = pick_s;
  }
  // b indexes the query groups (queries, block KV, outputs); groups of one
  // sequence share its context
  const int bc = b / groups;
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int pipe = wv / NWP, w = wv % NWP;
  const int tid = threadIdx.x % NTH, lane = threadIdx.x & 63, q4 = lane >> 4, l16 = lane & 15;
  const int64_t n_ctx = kv_len(ctx, bc);
  const int64_t n_keys = n_ctx + block;
  const int64_t k_begin = (int64_t)split * keys_per_split;
  const int64_t k_end = min(k_begin + (int64_t)keys_per_split, n_keys);
  // The split's keys are tiled in two runs: context rows [c_lo, c_hi) and the
  // block's own rows [r_lo, r_hi) (block row indices); every tile then has a
  // uniform base, a uniform row stride and a count of valid rows.
  const int64_t c_lo = k_begin, c_hi = min(k_end, n_ctx);
  const int ntc = c_hi > c_lo ? (int)((c_hi - c_lo + KT - 1) / KT) : 0;
  const int64_t r_lo = max(k_begin, n_ctx) - n_ctx, r_hi = k_end - n_ctx;
  const int ntb = r_hi > r_lo ? (int)((r_hi - r_lo + KT - 1) / KT) : 0;
  const int ntile = ntc + ntb;
  const int rounds = (ntile + P - 1) / P;
  char *ring = smem + pipe * 2 * STAGE;

  // ---- query fragments (loaded first: their wait below leaves the tile
  // prefetch issued after them in flight)
  const int rbase = mblk * (NWP * RW) + w * RW;
  bf16x8 qf[CB][NKS];
  int64_t qoff[CB];
  bool rvalid[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int r = rbase + 16 * cb + l16;
    rvalid[cb] = r < M;
    const int g = rvalid[cb] ? r / block : 0, i = rvalid[cb] ? r % block : 0;
    qoff[cb] = (((int64_t)b * block + i) * Hq + h * G + g) * D;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[cb][ks] = rvalid[cb] ? as_bf16x8(ldg16(q + qoff[cb] + 32 * ks + 8 * q4))
                              : as_bf16x8(make_uint4(0u, 0u, 0u, 0u));
  }

  // ---- tile addressing: chunk u of this thread is row x / CPR, chunk x % CPR
  // with x = tid + u * NTH, for K and V alike
  const int64_t crs = ctx.ss * 2;             // context row stride (bytes)
  const int64_t brs = (int64_t)Hkv * D * 2;   // block row stride (bytes)
  const char *ckb = ctx.k + ((int64_t)bc * ctx.sb + (int64_t)h * ctx.sh) * 2;
  const char *cvb = ctx.v + ((int64_t)bc * ctx.sb + (int64_t)h * ctx.sh) * 2;
  const char *bkb = reinterpret_cast<const char *>(blk_k) + ((int64_t)b * block * Hkv + h) * D * 2;
  const char *bvb = reinterpret_cast<const char *>(blk_v) + ((int64_t)b * block * Hkv + h) * D * 2;
  // Tile `it` of this pipeline (tile index it * P + pipe): K and V bases, row
  // stride and valid rows (0 past the split's last tile, whose rows are then
  // read from the last tile, in bounds, and masked).
  struct Tile {
    const char *k, *v;
    int64_t r0;       // first context row (context tiles)
    int stride, nvalid;
    bool in_ctx;
  };
  auto tile = [&](int it) {
    int t = it * P + pipe;
    const bool live = t < ntile;
    t = live ? t : (ntile > 0 ? ntile - 1 : 0);
    Tile d;
    d.in_ctx = t < ntc;
    if (t < ntc) {
      const int64_t r0 = c_lo + (int64_t)t * KT;
      d.r0 = r0;
      d.k = ckb + r0 * crs;
      d.v = cvb + r0 * crs;
      d.stride = (int)crs;
      d.nvalid = (int)min((int64_t)KT, c_hi - r0);
    } else {
      // (a split with no keys at all reads block row 0, masked)
      const int64_t r0 = ntile > 0 ? r_lo + (int64_t)(t - ntc) * KT : 0;
      d.r0 = 0;
      d.k = bkb + r0 * brs;
      d.v = bvb + r0 * brs;
      d.stride = (int)brs;
      d.nvalid = ntile > 0 ? (int)min((int64_t)KT, r_hi - r0) : 1;
    }
    d.nvalid = live ? d.nvalid : 0;
    return d;
  };
  uint4 kr[2][LPT], vr[2][LPT];
  auto fetch = [&](uint4 (&kx)[LPT], uint4 (&vx)[LPT], int it) {
    const Tile d = tile(it);
    const int last = d.nvalid > 0 ? d.nvalid - 1 : 0;
    if (PAGED && d.in_ctx) {  // context rows through the page table
#pragma unroll
      for (int u = 0; u < LPT; ++u) {
        const int x = tid + u * NTH;
        const int64_t e = kv_row(ctx, bc, h, d.r0 + min(x / CPR, last)) * 2 + (x % CPR) * 16;
        kx[u] = ldg16(ctx.k + e);
        vx[u] = ldg16(ctx.v + e);
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
      const int x = tid + u * NTH;
      const uint32_t off = (uint32_t)(min(x / CPR, last) * d.stride + (x % CPR) * 16);
      kx[u] = ldg16(d.k + off);
      vx[u] = ldg16(d.v + off);
    }
  };
  // registers -> LDS stage `stg` (swizzled row-major K and V)
  auto stash = [&](const uint4 (&kx)[LPT], const uint4 (&vx)[LPT], int stg) {
    char *Ks = ring + stg * STAGE, *Vs = Ks + KB;
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
      const int x = tid + u * NTH;
      const int row = x / CPR, c = x % CPR;
      const int fk = (row >> RSH) & (CPR - 1);
      const int fv = 2 * ((row >> RSH) & (CPR / 2 - 1));
      *reinterpret_cast<uint4 *>(Ks + row * ROWB + 16 * (c ^ fk)) = kx[u];
      *reinterpret_cast<uint4 *>(Vs + row * ROWB + 16 * (c ^ fv)) = vx[u];
    }
  };

  // o[cb][NDB] accumulates the softmax denominator (a block of ones times P^T)
  f32x4 o[CB][NDB + 1];
  float m_run[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    m_run[cb] = -INFINITY;  // reference max of raw scores
#pragma unroll
    for (int db = 0; db <= NDB; ++db) o[cb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const bf16x8 ones = as_bf16x8(make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u));
  // LDS read offsets inside a stage. K: row 16 kb + l16, chunk 4 ks + q4.
  // Transposed V: this lane supplies the address of row 16 hv + 4 q4 + l16 / 4,
  // d = 16 db + 4 (l16 % 4), i.e. chunk 2 db + (l16 % 4) / 2, byte 8 (l16 % 2).
  int kofs[2][NKS];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int row = 16 * kb + l16;
      kofs[kb][ks] = row * ROWB + 16 * ((4 * ks + q4) ^ ((row >> RSH) & (CPR - 1)));
    }
  int vofs[2], vf[2];
#pragma unroll
  for (int hv = 0; hv < 2; ++hv) {
    const int row = 16 * hv + 4 * q4 + (l16 >> 2);
    vofs[hv] = KB + row * ROWB + 8 * (l16 & 1);
    vf[hv] = 2 * ((row >> RSH) & (CPR / 2 - 1));
  }
  const int vchk = (l16 & 3) >> 1;

  auto compute = [&](int it) {
    const int nvalid = tile(it).nvalid;
    const char *stg = ring + (it & 1) * STAGE;
    // S^T (keys x queries), one 16-key block at a time; lane (l16, q4)
    // holds keys 16 kb + 4 q4 + j of query column l16 of each column block
    f32x4 s[2][CB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 a[NKS];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        a[ks] = as_bf16x8(*reinterpret_cast<const uint4 *>(stg + kofs[kb][ks]));
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        s[kb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
          s[kb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], qf[cb][ks], s[kb][cb], 0, 0, 0);
      }
    }
    if (nvalid < KT) {      // partial (or, past the split's end, empty) tile
      asm volatile("");     // keep this a branch: full tiles skip it
      const int lim = nvalid;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (16 * kb + 4 * q4 + j >= lim) s[kb][cb][j] = -INFINITY;
    }
    // online softmax on raw scores; the scale and log2(e) enter through one
    // FMA in the exp2 argument. Lazy rescaling: the reference max moves only
    // when a row's max exceeds it by more than 2^8 in probability (or on the
    // first tile); probabilities up to 256 are accumulated against the old
    // reference, which bf16 P and fp32 O hold exactly as well.
    bf16x8 pb[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      float mx = s[0][cb][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) mx = fmaxf(mx, s[kb][cb][j]);
      mx = max4q(mx);
      if (__ballot((mx - m_run[cb]) * sl2 > 8.f)) {
        const float m_new = fmaxf(m_run[cb], mx);
        const float alpha = __builtin_amdgcn_exp2f((m_run[cb] - m_new) * sl2);
#pragma unroll
        for (int db = 0; db <= NDB; ++db) o[cb][db] *= alpha;
        m_run[cb] = m_new;
      }
      // (a pipeline whose tiles were all empty so far has no reference yet;
      // its fully masked scores then give exp2(-inf) = 0)
      const float nb = m_run[cb] == -INFINITY ? 0.f : -m_run[cb] * sl2;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          s[kb][cb][j] = __builtin_amdgcn_exp2f(fmaf(s[kb][cb][j], sl2, nb));
      // B operand slots 0..3: keys 4 q4 + j; slots 4..7: keys 16 + 4 q4 + j
      uint4 pw;
      pw.x = pack2(s[0][cb][0], s[0][cb][1]);
      pw.y = pack2(s[0][cb][2], s[0][cb][3]);
      pw.z = pack2(s[1][cb][0], s[1][cb][1]);
      pw.w = pack2(s[1][cb][2], s[1][cb][3]);
      pb[cb] = as_bf16x8(pw);
    }
    // O^T += V^T P^T: the A operand of d-block db is read transposed from the
    // row-major V tile, in the key order of the B slots above
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int c = 2 * db + vchk;
      const uint2 lo = lds_tr16(stg + vofs[0] + 16 * (c ^ vf[0]));
      const uint2 hi = lds_tr16(stg + vofs[1] + 16 * (c ^ vf[1]));
      const bf16x8 av = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        o[cb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb[cb], o[cb][db], 0, 0, 0);
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
      o[cb][NDB] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[cb], o[cb][NDB], 0, 0, 0);
  };

  // Prologue: tiles 0 and 1 into the two register sets, tile 0 into LDS
  // stage 0, tile 2 into the set it freed. Fetches and stashes run for every
  // round, also past this pipeline's last tile (those re-read the split's
  // last row, in bounds, and are never consumed): the number of loads in
  // flight is then the same on every path, which lets the compiler wait for
  // exactly the set being stashed and keep the other one in flight.
  fetch(kr[0], vr[0], 0);
  fetch(kr[1], vr[1], 1);
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) asm volatile("" ::"v"(qf[cb][ks]));
  stash(kr[0], vr[0], 0);
  fetch(kr[0], vr[0], 2);
  lds_barrier();
  // Round it: tile it + 1 (register set (it + 1) & 1) goes to LDS stage
  // (it + 1) & 1, tile it + 3 is fetched into that set, tile it is consumed
  // from stage it & 1. The loop is unrolled by two so that the register sets
  // are named statically.
  // The two waves that share a SIMD belong to pipelines p and p + P / 2; the
  // first half of the pipelines computes before it stashes and fetches, the
  // second half after, so that one wave's MFMA work meets the other's memory
  // and VALU work instead of the same unit.
  const bool compute_first = pipe < P / 2;
  auto round = [&](int it, uint4 (&kn)[LPT], uint4 (&vn)[LPT]) {
    if (compute_first) compute(it);
    stash(kn, vn, (it + 1) & 1);
    fetch(kn, vn, it + 3);
    if (!compute_first) compute(it);
    lds_barrier();
  };
  // (an odd round count gets one idle round: both halves of the unrolled body
  // always run, so the loads in flight at the loop head are the same on
  // every path into it)
  for (int it = 0; it < rounds; it += 2) {
    round(it, kr[1], vr[1]);
    round(it + 1, kr[0], vr[0]);
  }

  // Merge of the P pipelines, spread over every wave: wave w of pipeline p
  // merges d-blocks [p * SL, (p + 1) * SL) of its query rows over the P
  // pipelines and writes them out. Its own share of those stays in
  // registers; through LDS each wave hands the other pipelines their d-blocks
  // ([pipeline][wave][cb][NX d-blocks][lane], 16 B each, the writer's own
  // slice left out) and its (max, sum) ([pipeline][wave][cb][lane]).
  constexpr int SL = NDB / P;   // d-blocks each wave merges and writes
  constexpr int NX = NDB - SL;  // d-blocks each wave hands over
  static_assert(SL * P == NDB, "d-blocks must split evenly over the pipelines");
  const int db0 = pipe * SL;
  f32x4 acc[CB][SL];
  float mrow[CB], lrow[CB];
  if constexpr (P > 1) {
    f32x4 *xo = reinterpret_cast<f32x4 *>(smem);
    float2 *xm = reinterpret_cast<float2 *>(smem + (size_t)P * NWP * CB * NX * 64 * 16);
    const int pw = pipe * NWP + w;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int q = db / SL;  // the pipeline that merges this d-block
        if (q != pipe)
          xo[((pw * CB + cb) * NX + db - (q > pipe ? SL : 0)) * 64 + lane] = o[cb][db];
      }
      xm[(pw * CB + cb) * 64 + lane] = make_float2(m_run[cb], o[cb][NDB][0]);
    }
    lds_barrier();
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      float2 ml[P];
#pragma unroll
      for (int pp = 0; pp < P; ++pp) ml[pp] = xm[((pp * NWP + w) * CB + cb) * 64 + lane];
      float mm = ml[0].x;
#pragma unroll
      for (int pp = 1; pp < P; ++pp) mm = fmaxf(mm, ml[pp].x);
      float l = 0.f;
#pragma unroll
      for (int sb = 0; sb < SL; ++sb) acc[cb][sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int pp = 0; pp < P; ++pp) {
        // (a pipeline that saw only masked keys has max -inf and adds nothing)
        const float sc =
            ml[pp].x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((ml[pp].x - mm) * sl2);
        l += sc * ml[pp].y;
        if (pp == pipe) {
#pragma unroll
          for (int sb = 0; sb < SL; ++sb) acc[cb][sb] += sc * o[cb][pp * SL + sb];
        } else {
          const int pos = db0 - (pipe > pp ? SL : 0);  // where pipeline pp put them
#pragma unroll
          for (int sb = 0; sb < SL; ++sb)
            acc[cb][sb] += sc * xo[(((pp * NWP + w) * CB + cb) * NX + pos + sb) * 64 + lane];
        }
      }
      mrow[cb] = mm;
      lrow[cb] = l;
    }
  } else {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
      for (int sb = 0; sb < SL; ++sb) acc[cb][sb] = o[cb][sb];
      mrow[cb] = m_run[cb];
      lrow[cb] = o[cb][NDB][0];
    }
  }
  // lane holds d = 16 (db0 + sb) + 4 q4 + j of query row rbase + 16 cb + l16
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    if (!rvalid[cb]) continue;
    const int r = rbase + 16 * cb + l16;
    if (nsplit == 1) {
      const float inv = 1.f / lrow[cb];
      uint16_t *orow = out + qoff[cb] + 16 * db0 + 4 * q4;
#pragma unroll
      for (int sb = 0; sb < SL; ++sb) {
        uint2 wd;
        wd.x = pack2(acc[cb][sb][0] * inv, acc[cb][sb][1] * inv);
        wd.y = pack2(acc[cb][sb][2] * inv, acc[cb][sb][3] * inv);
        *reinterpret_cast<uint2 *>(orow + 16 * sb) = wd;
      }
    } else {
      const int64_t pidx = ((int64_t)b * Hkv + h) * nsplit + split;
      float *po = part_o + (pidx * M + r) * D + 16 * db0 + 4 * q4;
#pragma unroll
      for (int sb = 0; sb < SL; ++sb)
        *reinterpret_cast<float4 *>(po + 16 * sb) =
            make_float4(acc[cb][sb][0], acc[cb][sb][1], acc[cb][sb][2], acc[cb][sb][3]);
      if (pipe == 0 && q4 == 0) part_ml[pidx * M + r] = make_float2(mrow[cb] * sl2, lrow[cb]);
    }
  }
}

// Merge of split-KV partials (log2-domain statistics), 8 outputs per thread.
__global__ __launch_bounds__(256) void attn_combine_kernel(
    const float *__restrict__ part_o, const float2 *__restrict__ part_ml,
    uint16_t *__restrict__ out, int block, int Hq, int Hkv, int G, int M, int D,
    int nsplit) {
  const int h = blockIdx.y, b = blockIdx.z;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int r = idx / (D / 8), d0 = (idx % (D / 8)) * 8;
  if (r >= M) return;
  const int64_t p0 = ((int64_t)b * Hkv + h) * nsplit;
  // part_ml holds (max * scale * log2(e), sum) per row and split. Splits are
  // read eight at a time with every load of a group issued before its
  // arithmetic; the sums run over the splits in index order.
  constexpr int GRP = 8;
  float mx = -INFINITY;
  for (int s0 = 0; s0 < nsplit; s0 += GRP) {
    float2 ml[GRP];
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      ml[u] = s0 + u < nsplit ? part_ml[(p0 + s0 + u) * M + r] : make_float2(-INFINITY, 0.f);
#pragma unroll
    for (int u = 0; u < GRP; ++u) mx = fmaxf(mx, ml[u].x);
  }
  float den = 0.f, n[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) n[e] = 0.f;
  for (int s0 = 0; s0 < nsplit; s0 += GRP) {
    float2 ml[GRP];
    float4 v[GRP][2];
#pragma unroll
    for (int u = 0; u < GRP; ++u) {
      const bool in = s0 + u < nsplit;
      const int64_t sp = p0 + (in ? s0 + u : 0);
      ml[u] = in ? part_ml[sp * M + r] : make_float2(-INFINITY, 0.f);
      const float4 *src = reinterpret_cast<const float4 *>(part_o + (sp * M + r) * D + d0);
      v[u][0] = src[0];
      v[u][1] = src[1];
    }
#pragma unroll
    for (int u = 0; u < GRP; ++u) {
      if (ml[u].x == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(ml[u].x - mx);
      den += ml[u].y * w;
      n[0] += v[u][0].x * w; n[1] += v[u][0].y * w; n[2] += v[u][0].z * w; n[3] += v[u][0].w * w;
      n[4] += v[u][1].x * w; n[5] += v[u][1].y * w; n[6] += v[u][1].z * w; n[7] += v[u][1].w * w;
    }
  }
  const float inv = 1.f / den;
  const int g = r / block, i = r % block;
  uint16_t *orow = out + (((int64_t)b * block + i) * Hq + h * G + g) * D + d0;
  uint4 w;
  w.x = pack2(n[0] * inv, n[1] * inv);
  w.y = pack2(n[2] * inv, n[3] * inv);
  w.z = pack2(n[4] * inv, n[5] * inv);
  w.w = pack2(n[6] * inv, n[7] * inv);
  *reinterpret_cast<uint4 *>(orow) = w;
}

// fp32 path: one wave per query row; lanes split the keys of a 64-key pass,
// then accumulate P V with the probabilities broadcast across the wave.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float *__restrict__ q, KvView ctx, const float *__restrict__ blk_k,
    const float *__restrict__ blk_v, float *__restrict__ out, int block, int Hq, int Hkv,
    int G, int M, float scale, int groups) {
  constexpr int ND = (D + 63) / 64;
  const int h = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= M) return;
  const int g = r / block, i = r % block;
  const int64_t qoff = (((int64_t)b * block + i) * Hq + h * G + g) * D;
  const int bc = b / groups;  // context sequence of this query group
  const int64_t n_ctx = kv_len(ctx, bc);
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
          row_ptr(ctx, ck, bk, bc, b, h, key, n_ctx, block, Hkv, D, 4));
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
          row_ptr(ctx, cv, bv, bc, b, h, j0 + jj, n_ctx, block, Hkv, D, 4));
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

// Workgroups the split-KV plan aims for: one per CU of the 256-CU gfx950
// (each workgroup takes a whole CU's registers). The plan is host-only (the
// workspace queries run without a device), so this is not read from the GPU.
constexpr int kTargetWgs = 256;

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
  // Row blocks of 64 rows: 4 pipelines of 2 waves x 32 rows (512 threads);
  // blocks of at most 32 rows: 4 pipelines of one wave.
  p.stages = 2;
  p.key_tile = 32;
  if (p.M > 32) {
    p.rows_per_wave = 32, p.nwaves = 2;
  } else {
    p.rows_per_wave = p.M > 16 ? 32 : 16, p.nwaves = 1;
  }
  const int64_t max_keys = max_ctx + block;
  const int64_t ntile = (max_keys + p.key_tile - 1) / p.key_tile;
  auto split_keys = [&](int pipes, int nwaves) {
    p.pipes = pipes;
    p.nwaves = nwaves;
    p.n_mblk = (p.M + p.rows_per_wave * p.nwaves - 1) / (p.rows_per_wave * p.nwaves);
    const int64_t base = (int64_t)batch * hd.num_kv_heads * p.n_mblk;
    // one workgroup per CU; every split gets at least one tile per pipeline
    int64_t want = (kTargetWgs + base - 1) / base;
    if (want < 1) want = 1;
    const int64_t most = (ntile + p.pipes - 1) / p.pipes;
    const int64_t ns = want < most ? want : most;
    const int64_t tiles_per = (ntile + ns - 1) / ns;
    p.keys_per_split = (int)(tiles_per * p.key_tile);
    p.nsplit = (int)((max_keys + p.keys_per_split - 1) / p.keys_per_split);
    // nsplit <= min(want, ceil(ntile / pipes)), which grows with the context:
    // sizing the partials by it covers every shorter context too
    p.nsplit_cap = (int)ns;
  };
  split_keys(4, p.nwaves);
  // When the keys are split anyway (and a combine runs), 128-row blocks (2
  // pipelines of 4 waves) read each KV head's keys once per split instead of
  // once per 64-row block. (A shorter context under the same shapes splits
  // at most as many ways, so partials sized by the longest one still fit.)
  if (p.M >= 128 && p.nsplit_cap > 1) split_keys(2, 4);
  if (p.nsplit_cap > 1) {
    const size_t parts = (size_t)batch * hd.num_kv_heads * p.nsplit_cap * p.M;
    p.part_o_bytes = parts * hd.head_dim * sizeof(float);
    p.part_ml_bytes = parts * sizeof(float2);
  }
  return p;
}

hipError_t launch_block_attn(const herald_heads &hd, int batch, int block, int groups,
                             const void *q, const KvView &ctx, int64_t max_ctx,
                             const void *blk_k, const void *blk_v, void *out, void *ws,
                             hipStream_t stream) {
  // the query groups of all sequences form one batch of batch * groups
  batch *= groups;
  const AttnPlan p = attn_plan(hd, batch, block, max_ctx);
  const int G = hd.num_q_heads / hd.num_kv_heads;
  const int Hq = hd.num_q_heads, Hkv = hd.num_kv_heads, D = hd.head_dim;
  if (hd.dtype != HERALD_BF16) {
    const dim3 grid(p.n_mblk, Hkv, batch);
    const float scale = (float)(1.0 / sqrt((double)D));
    if (D == 64)
      attn_f32_kernel<64><<<grid, 256, 0, stream>>>(
          (const float *)q, ctx, (const float *)blk_k, (const float *)blk_v, (float *)out,
          block, Hq, Hkv, G, p.M, scale, groups);
    else if (D == 128)
      attn_f32_kernel<128><<<grid, 256, 0, stream>>>(
          (const float *)q, ctx, (const float *)blk_k, (const float *)blk_v, (float *)out,
          block, Hq, Hkv, G, p.M, scale, groups);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  char *w = reinterpret_cast<char *>(ws);
  float *part_o = reinterpret_cast<float *>(w);
  float2 *part_ml = reinterpret_cast<float2 *>(w + ((p.part_o_bytes + 255) & ~(size_t)255));
  const float sl2 = (float)(1.0 / sqrt((double)D)) * kLog2e;
  const int grid = batch * Hkv * p.nsplit * p.n_mblk;
  const uint16_t *qq = (const uint16_t *)q;
  const uint16_t *bk = (const uint16_t *)blk_k, *bv = (const uint16_t *)blk_v;
  uint16_t *oo = (uint16_t *)out;
  const bool paged = ctx.pt != nullptr;
  // Longest context first when the workgroups do not all fit at once and
  // each covers enough keys (from 1024, tens of microseconds of work) that
  // ranking the query groups (about a microsecond per workgroup) is small
  // beside the idle tail of a ragged batch it removes.
  const int order =
      grid > kTargetWgs && batch > 1 && batch <= kOrderMax && max_ctx + block >= 1024;
#define HERALD_ATTN(D_, RW_, NW_, P_, PG_)                                               \
  if (D == D_ && p.rows_per_wave == RW_ && p.nwaves == NW_ && p.pipes == P_ &&            \
      paged == PG_) {                                                                    \
    auto kfn = attn_bf16_kernel<D_, RW_, NW_, P_, PG_>;                                   \
    constexpr int kSmem = attn_smem_bytes<D_, RW_, NW_, P_>();                            \
    static const hipError_t attr_err = hipFuncSetAttribute(                               \
        reinterpret_cast<const void *>(kfn), hipFuncAttributeMaxDynamicSharedMemorySize,  \
        kSmem);                                                                          \
    if (attr_err != hipSuccess) return attr_err;                                         \
    kfn<<<grid, NW_ * P_ * 64, kSmem, stream>>>(qq, ctx, bk, bv, oo, part_o, part_ml,     \
                                               block, Hq, Hkv, G, p.M, p.n_mblk,         \
                                               p.nsplit, p.keys_per_split, sl2, groups,  \
                                               order);                                   \
  } else
  HERALD_ATTN(64, 32, 2, 4, false) HERALD_ATTN(64, 32, 1, 4, false)
  HERALD_ATTN(64, 16, 1, 4, false) HERALD_ATTN(64, 32, 4, 2, false)
  HERALD_ATTN(128, 32, 2, 4, false) HERALD_ATTN(128, 32, 1, 4, false)
  HERALD_ATTN(128, 16, 1, 4, false) HERALD_ATTN(128, 32, 4, 2, false)
  HERALD_ATTN(64, 32, 2, 4, true) HERALD_ATTN(64, 32, 1, 4, true)
  HERALD_ATTN(64, 16, 1, 4, true) HERALD_ATTN(64, 32, 4, 2, true)
  HERALD_ATTN(128, 32, 2, 4, true) HERALD_ATTN(128, 32, 1, 4, true)
  HERALD_ATTN(128, 16, 1, 4, true) HERALD_ATTN(128, 32, 4, 2, true)
  return hipErrorInvalidValue;
#undef HERALD_ATTN
  if (p.nsplit > 1) {
    const dim3 cg((p.M * (D / 8) + 255) / 256, Hkv, batch);
    attn_combine_kernel<<<cg, 256, 0, stream>>>(part_o, part_ml, oo, block, Hq, Hkv, G,
                                                p.M, D, p.nsplit);
  }
  return hipGetLastError();
}

}  // namespace herald
