// Selection phase on gfx950: representative query, full-cache scoring, GQA
// importance and per-KV-head top-k (sec. IV-A.2 and sec. IV-B.4 of the paper).
//
// Four launches per call, all on the caller's stream:
//   repq   : qbar[b][h][e][g] = mean over the B block queries (fp64), one
//            (element, head) per thread, and clears the first-level histogram.
//   score  : one workgroup per (chunk of 2048 cached rows, KV head, sequence).
//            Streams K once with coalesced 128-bit non-temporal loads and
//            forms the G raw scores of every row in fp64: on the fp64 matrix
//            cores for G <= 4 (each wave stages its tiles through its own LDS
//            region into the MFMA operand layout), with fp64 FMAs for G = 8.
//            Writes the scores z (fp64) and the chunk's softmax statistics
//            (max, sum of exp).
//   norm   : merges the chunk statistics into (m_g, l_g), forms the GQA
//            importance s_hat = sum_g exp(z_g - m_g) / l_g (fp64), stores its
//            bit pattern as a 64-bit ranking key, and histograms the key's
//            exponent field.
//   topk   : one workgroup per (KV head, sequence). MSB-first radix select on
//            the 64-bit keys (exponent from the histogram, then 11-bit digits;
//            once the boundary bucket fits, it is compacted into LDS), then an
//            ordered emission pass that writes the selected indices ascending,
//            taking equal keys lowest index first.
// Identical scores give bit-identical importances (one shift m_g per head for
// every row), so exact ties are decided by index, as the definition says.
//
// Selection with x query rows (herald_select_xq) replaces repq by rows (the x
// centred block rows converted to fp64) and, for more than 4 score rows
// (query row, head) per KV head, score and norm by score_rows and norm_rows;
// top-k is the same.
#include <math.h>

#include "common.h"
#include "select.h"

namespace herald {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kCandCap = 16384;  // LDS candidates (128 KiB of keys)
constexpr int kKeysPerThread = 16;  // keys per thread and round in the passes over S

// (m, l) <- softmax-statistics merge of (m, l) and (m2, l2).
__device__ __forceinline__ void merge_ml(double &m, double &l, double m2, double l2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) { m = m2; l = l2; return; }
  if (m2 > m) { l = l * exp(m - m2) + l2; m = m2; }
  else { l += l2 * exp(m2 - m); }
}

// (m, 1 / l) of score row v of (b, h) over the whole cache and the tail:
// the nch chunk partials, then the tail slot, merged by one wave in a fixed
// order (lower lane first), so that every caller, in every lane, gets
// bit-identical values.
__device__ __forceinline__ void merged_stats(const double *__restrict__ part, int64_t bh,
                                             int nslot, int nch, int V, int v, int lane,
                                             double &m_out, double &inv_out) {
  double m = -INFINITY, l = 0.0;
  for (int c = lane; c <= nch; c += 64) {
    const int slot = c < nch ? c : nslot - 1;  // the chunks, then the tail
    const double *p = part + ((bh * nslot + slot) * V + v) * 2;
    merge_ml(m, l, p[0], p[1]);
  }
#pragma unroll
  for (int off = 1; off <= 32; off <<= 1) {
    const double m2 = __shfl_xor(m, off, 64);
    const double l2 = __shfl_xor(l, off, 64);
    if (lane & off) { double tm = m2, tl = l2; merge_ml(tm, tl, m, l); m = tm; l = tl; }
    else merge_ml(m, l, m2, l2);
  }
  m_out = m;
  inv_out = 1.0 / l;
}

// ---------------------------------------------------------------- repq
template <int D, int G, bool BF16>
__global__ __launch_bounds__(256) void repq_kernel(const void *__restrict__ q_sel,
                                                   double *__restrict__ qbar,
                                                   uint32_t *__restrict__ hist,
                                                   double *__restrict__ part, int nslot,
                                                   int block, int Hq, int Hkv) {
  constexpr int U = 64;  // loads in flight per thread: every block row at once
  const int h = blockIdx.x, b = blockIdx.y;
  const int64_t bh = (int64_t)b * Hkv + h;
  // one (element, head) per thread; blockIdx.z covers the D * G of them
  const int t = blockIdx.z * 256 + threadIdx.x;
  if (t < D * G) {
    const int e = t % D, g = t / D;
    const int hq = h * G + g;
    const int64_t base = ((int64_t)b * block * Hq + hq) * D + e;
    const int64_t step = (int64_t)Hq * D;
    double acc = 0.0;
    for (int i0 = 0; i0 < block; i0 += U) {
      // every load is issued (rows past the block re-read its last row) so
      // that all of them are in flight together; the sum takes only the
      // block's rows, in block-row order
      float x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = min(i0 + u, block - 1);
        if (BF16)
          x[u] = __uint_as_float(
              (uint32_t)reinterpret_cast<const uint16_t *>(q_sel)[base + i * step] << 16);
        else
          x[u] = reinterpret_cast<const float *>(q_sel)[base + i * step];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)  // (past the block: + 0.0, which leaves acc as is)
        acc += i0 + u < block ? (double)x[u] : 0.0;
    }
    qbar[(bh * D + e) * G + g] = acc / (double)block;
  }
  if (blockIdx.z == 0) {
    for (int i = threadIdx.x; i < kHistBins; i += 256) hist[bh * kHistBins + i] = 0u;
    // no normalisation tail unless tail_kernel fills its slot
    if (threadIdx.x < G) {
      double *p = part + ((bh * nslot + nslot - 1) * G + threadIdx.x) * 2;
      p[0] = -INFINITY;
      p[1] = 0.0;
    }
  }
}

// ---------------------------------------------------------------- score (FMA)
// Used for G = 8. Workgroup = 2 wave pairs. A pair scores one 64-row tile at a time: both
// waves stage the tile (coalesced 1 KiB loads) into LDS, then each lane owns
// one row and each wave of the pair forms the partial dot products of one
// half of the head dimension with the qbar half it holds in scalar registers.
// The halves are added in a fixed order (low half + high half); the online
// softmax statistics of the G heads are split between the two waves.
// (chunk, KV head, sequence) of a workgroup of a (chunk, H_kv, batch) grid,
// numbered chunk-major. Workgroups are dealt to the 8 XCDs round-robin by
// linear id; numbered chunk-fastest, the low chunks that every sequence has
// would all land on the same few XCDs when the sequences' lengths differ,
// while with the chunk as the slowest index the (KV head, sequence) pairs
// alternate over the XCDs and each gets an equal share of the valid chunks.
struct ChunkOf {
  int chunk, h, b;
};
__device__ __forceinline__ ChunkOf chunk_major() {
  const int64_t nbh = (int64_t)gridDim.y * gridDim.z;
  const int64_t lin =
      blockIdx.x + (int64_t)gridDim.x * (blockIdx.y + (int64_t)gridDim.y * blockIdx.z);
  ChunkOf c;
  c.chunk = (int)(lin / nbh);
  const int bhi = (int)(lin - (int64_t)c.chunk * nbh);
  c.h = bhi % (int)gridDim.y;
  c.b = bhi / (int)gridDim.y;
  return c;
}

// Page numbers of the pages that hold rows [c0, c0 + kScoreChunk) of
// sequence b, staged in LDS by the workgroup (paged views): a tile's page
// lookup is then an LDS read instead of a global load that its row loads wait
// for. Pages hold at least 8 rows, so a chunk spans at most kChunkPages pages;
// entries of pages past the sequence's rows (never read) are 0.
constexpr int kChunkPages = kScoreChunk / 8;
__device__ __forceinline__ void stage_chunk_pages(const KvView &kv, int b, int64_t c0,
                                                  int64_t S, int32_t *spt) {
  const int shift = kv.page_shift;
  const int64_t p0 = c0 >> shift;
  const int n = shift >= 11 ? 1 : (kScoreChunk >> shift);
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int64_t pg = p0 + i;
    spt[i] = pg < kv.max_pages && (pg << shift) < S ? kv.pt[(int64_t)b * kv.max_pages + pg] : 0;
  }
  __syncthreads();
}

template <int D, int G, bool BF16, bool PAGED>
__global__ __launch_bounds__(256, 4) void score_kernel(KvView kv,
                                                       const double *__restrict__ qbar,
                                                       double *__restrict__ zspill,
                                                       double *__restrict__ part,
                                                       int Hkv, int64_t S_pad,
                                                       int nslot, double scale) {
  constexpr int ELT = BF16 ? 2 : 4;
  constexpr int RB = D * ELT;         // bytes per cached row
  constexpr int LPR = RB / 16;        // lanes per row in one 1 KiB load
  constexpr int RPL = 64 / LPR;       // rows per 1 KiB load
  constexpr int NLD = LPR;            // 1 KiB loads per 64-row tile
  constexpr int NLDW = NLD / 2;       // loads per wave of the pair
  constexpr int LSTR = RB + 16;       // padded LDS row stride
  constexpr int EPC = 16 / ELT;       // elements per 16-byte chunk
  constexpr int HB = RB / 2;          // bytes of one half row
  constexpr int NCH = HB / 16;        // 16-byte chunks per half row
  constexpr int GH = G > 1 ? G / 2 : 1;  // heads whose statistics a wave keeps
  constexpr int NTP = kScoreChunk / 128; // tiles per pair
  __shared__ __attribute__((aligned(16))) char lds[2 * 64 * LSTR];
  __shared__ double xch[2][2][64][GH];   // [pair][from half][row][g]
  __shared__ double red[4][GH], red2[4][GH];

  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t S = kv_len(kv, b);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  // wave index made provably uniform, so that qbar addresses stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int pair = wave >> 1, half = wave & 1;
  char *my = lds + pair * 64 * LSTR;
  const int64_t bh = (int64_t)b * Hkv + h;
  // qbar layout [e][g]; this wave's half of the elements
  const double *qb = qbar + bh * D * G + (size_t)half * (D / 2) * G;
  const int lr = lane / LPR, lc = lane % LPR;
  const char *kbase = kv.k + ((int64_t)b * kv.sb + (int64_t)h * kv.sh) * ELT + lc * 16;
  // heads whose statistics this wave keeps: [g0, g0 + GH)
  const int g0 = G > 1 ? half * GH : 0;
  const bool keeps = G > 1 || half == 0;

  __shared__ int32_t spt[PAGED ? kChunkPages : 1];
  if constexpr (PAGED) stage_chunk_pages(kv, b, c0, S, spt);
  auto row_addr = [&](int64_t s_base, int64_t s) -> const char * {
    if (PAGED) {
      const int64_t page = spt[(s_base >> kv.page_shift) - (c0 >> kv.page_shift)];
      return kv.k + (page * kv.sp + (int64_t)h * kv.sh +
                     (s & ((1 << kv.page_shift) - 1)) * kv.ss) * ELT + lc * 16;
    }
    return kbase + s * kv.ss * ELT;
  };
  auto tile_row0 = [&](int t) { return c0 + (int64_t)(2 * t + pair) * 64; };

  uint4 buf[NLDW];
  auto load_tile = [&](int t) {
    const int64_t r0 = tile_row0(t) + half * (NLDW * RPL);
    if (r0 + NLDW * RPL <= S) {
#pragma unroll
      for (int i = 0; i < NLDW; ++i)
        buf[i] = ldg16_nt(row_addr(r0 + i * RPL, r0 + i * RPL + lr));
    } else {
#pragma unroll
      for (int i = 0; i < NLDW; ++i) {
        const int64_t s = r0 + i * RPL + lr;
        buf[i] = make_uint4(0u, 0u, 0u, 0u);
        if (s < S) buf[i] = ldg16_nt(row_addr(r0 + i * RPL, s));
      }
    }
  };

  double m_l[GH], l_l[GH];
#pragma unroll
  for (int g = 0; g < GH; ++g) { m_l[g] = -INFINITY; l_l[g] = 0.0; }
  load_tile(0);
#pragma unroll 1
  for (int t = 0; t < NTP; ++t) {
    if (c0 + (int64_t)(2 * t) * 64 >= S) break;  // uniform: rest of chunk is empty
#pragma unroll
    for (int i = 0; i < NLDW; ++i)
      *reinterpret_cast<uint4 *>(my + (half * NLDW * RPL + i * RPL + lr) * LSTR + lc * 16) =
          buf[i];
    __syncthreads();
    if (t + 1 < NTP) load_tile(t + 1);
    double acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.0;
    // two 16-byte chunks per step: enough to overlap the LDS and scalar
    // loads, few enough that the fp64 operands fit in registers
#pragma unroll 2
    for (int j = 0; j < NCH; ++j) {
      const uint4 c = *reinterpret_cast<const uint4 *>(my + lane * LSTR + half * HB + j * 16);
      // A uniform zero the compiler cannot see through keeps the qbar loads
      // in scalar registers, a chunk at a time, instead of hoisting them all.
      int zero = 0;
      asm volatile("" : "+s"(zero));
      const double *qq = qb + zero + j * EPC * G;
      const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (BF16) {
          const double x0 = (double)bf16_lo(w[u]);
          const double x1 = (double)bf16_hi(w[u]);
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] = fma(x0, qq[(2 * u) * G + g], acc[g]);
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] = fma(x1, qq[(2 * u + 1) * G + g], acc[g]);
        } else {
          const double x = (double)__uint_as_float(w[u]);
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] = fma(x, qq[u * G + g], acc[g]);
        }
      }
    }
    // hand the partials of the other wave's heads over
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int owner = G > 1 ? g / GH : 0;
      if (owner != half) xch[pair][half][lane][g % GH] = acc[g];
    }
    __syncthreads();
    const int64_t s = tile_row0(t) + lane;
    if (keeps && s < S) {
      double *dst = zspill + (bh * S_pad + s) * G;
#pragma unroll
      for (int gg = 0; gg < GH; ++gg) {
        const int g = g0 + gg;
        const double other = xch[pair][half ^ 1][lane][gg];
        const double z = (half == 0 ? acc[g] + other : other + acc[g]) * scale;
        dst[g] = z;
        // one exp per score: exp(-|z - m|) either rescales the old sum or
        // is the new term
        const double dz = z - m_l[gg];
        const double e = exp(-fabs(dz));
        const bool up = dz > 0.0;
        l_l[gg] = up ? fma(l_l[gg], e, 1.0) : l_l[gg] + e;
        m_l[gg] = up ? z : m_l[gg];
      }
    }
  }

  // chunk statistics: max over the workgroup, then the rescaled sums. Waves
  // w and w ^ 2 (same half) keep the same heads.
#pragma unroll
  for (int gg = 0; gg < GH; ++gg) {
    double m = m_l[gg];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
    if (lane == 0) red[wave][gg] = m;
  }
  __syncthreads();
  double mc[GH];
#pragma unroll
  for (int gg = 0; gg < GH; ++gg) mc[gg] = fmax(red[half][gg], red[half + 2][gg]);
#pragma unroll
  for (int gg = 0; gg < GH; ++gg) {
    double v = m_l[gg] == -INFINITY ? 0.0 : l_l[gg] * exp(m_l[gg] - mc[gg]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    if (lane == 0) red2[wave][gg] = v;
  }
  __syncthreads();
  if (wave < 2 && lane < GH && (G > 1 || wave == 0)) {
    const int gg = lane, g = g0 + gg;
    double *p = part + ((bh * nslot + chunk) * G + g) * 2;
    p[0] = fmax(red[half][gg], red[half + 2][gg]);
    p[1] = red2[half][gg] + red2[half + 2][gg];
  }
}

// ---------------------------------------------------------------- score (MFMA)
// The dot products run on the fp64 matrix cores: v_mfma_f64_4x4x4_4b forms
// four independent 4x4x4 products per instruction. Each of its blocks takes
// four cached rows (A: 4 rows x 4 head-dim elements) against the same qbar
// slice (B: 4 elements x the query heads of the group, zero past G), so a
// chain of D/4 instructions scores 16 rows for all G heads, every multiply
// useful when G = 4. Operand layout: A lane l holds row l % 16 at element
// slot l / 16, B lane l holds slot l / 16 of head l % 4, and the result of
// lane l is row 4 ((l / 4) % 4) + l / 16, head l % 4. The head dimension is
// enumerated in the same permuted order on both operands (a sum does not
// depend on it beyond rounding) so that a lane reads whole 16-byte pieces of
// its row. Two accumulators per 16 rows (first and second half of the
// elements, added in that order) and up to four 16-row chains per tile keep
// independent chains in flight.
// Each wave scores its own 8 KiB tiles (64, 32 or 16 rows of 128, 256 or 512
// bytes): coalesced 1 KiB loads into a
// wave-private LDS region, read back in the operand layout; the next tile's
// loads are in flight while the current one is multiplied. The only
// workgroup barriers merge the chunk statistics at the end.
template <int D, int G, bool BF16, bool PAGED>
__global__ __launch_bounds__(256, 2) void score_mfma_kernel(KvView kv,
                                                            const double *__restrict__ qbar,
                                                            double *__restrict__ zspill,
                                                            double *__restrict__ part,
                                                            int Hkv, int64_t S_pad,
                                                            int nslot, double scale) {
  static_assert(G <= 4, "one MFMA column per query head of the group");
  constexpr int ELT = BF16 ? 2 : 4;
  constexpr int RB = D * ELT;                   // bytes per cached row
  constexpr int EPP = 16 / ELT;                 // elements per 16-byte piece
  constexpr int NP = RB / 64;                   // pieces per lane and row (4 lanes per row)
  constexpr int NS = D / 4;                     // MFMA steps over the head dimension
  constexpr int NH = NS / 2;                    // steps per accumulator
  constexpr int WR = 8192 / RB;                 // rows per wave tile
  constexpr int NC = WR / 16;                   // 16-row chains per tile
  constexpr int RPL = 1024 / RB;                // rows per wave-wide 1 KiB load
  constexpr int LPR = RB / 16;                  // lanes per row in such a load
  constexpr int NLD = WR / RPL;                 // loads per lane and tile
  constexpr int LSTR = RB + 16;                 // padded LDS row stride
  constexpr int NW = 4;                         // waves per workgroup
  constexpr int TPW = kScoreChunk / (WR * NW);  // tiles per wave
  static_assert(NP * EPP == NS && NS % 2 == 0, "head dimension split");
  __shared__ __attribute__((aligned(16))) char lds[NW][WR * LSTR];
  __shared__ double red[NW][4], red2[NW][4];

  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t S = kv_len(kv, b);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t bh = (int64_t)b * Hkv + h;
  char *my = lds[wave];
  const int kq = lane >> 4;                               // element slot (A and B)
  const int g = lane & 3;                                 // head (B column, result)
  const int zrow = 4 * ((lane >> 2) & 3) + (lane >> 4);   // result row within 16

  // B operand of every step: qbar at the permuted element, zero past G,
  // in LDS as [step][slot kq][head g] (the lanes of one (kq, g) share it)
  __shared__ double bqs[NS * 16];
  for (int i = threadIdx.x; i < NS * 16; i += 256) {
    const int s = i >> 4, kk = (i >> 2) & 3, gg = i & 3;
    const int e = (s / EPP) * (4 * EPP) + kk * EPP + s % EPP;
    bqs[i] = gg < G ? qbar[(bh * D + e) * G + gg] : 0.0;
  }
  __syncthreads();
  const double *bql = bqs + kq * 4 + g;

  const int lr = lane / LPR, lc = lane % LPR;
  const char *kbase = kv.k + ((int64_t)b * kv.sb + (int64_t)h * kv.sh) * ELT + lc * 16;
  // row s of a load whose first row s_base is uniform (a load never crosses
  // a page: pages hold at least 8 rows and loads start at multiples of RPL)
  __shared__ int32_t spt[PAGED ? kChunkPages : 1];
  if constexpr (PAGED) stage_chunk_pages(kv, b, c0, S, spt);
  auto row_addr = [&](int64_t s_base, int64_t s) -> const char * {
    if (PAGED) {
      const int64_t page = spt[(s_base >> kv.page_shift) - (c0 >> kv.page_shift)];
      return kv.k + (page * kv.sp + (int64_t)h * kv.sh +
                     (s & ((1 << kv.page_shift) - 1)) * kv.ss) * ELT + lc * 16;
    }
    return kbase + s * kv.ss * ELT;
  };
  // the waves take interleaved tiles, so that together they stream the chunk
  auto tile_row0 = [&](int t) { return c0 + (int64_t)(t * NW + wave) * WR; };
  uint4 buf[NLD];
  auto load_tile = [&](int t) {
    const int64_t r0 = tile_row0(t);
    if (r0 + WR <= S) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) buf[i] = ldg16_nt(row_addr(r0 + i * RPL, r0 + i * RPL + lr));
    } else {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const int64_t s = r0 + i * RPL + lr;
        buf[i] = make_uint4(0u, 0u, 0u, 0u);
        if (s < S) buf[i] = ldg16_nt(row_addr(r0 + i * RPL, s));
      }
    }
  };

  double m_l = -INFINITY, l_l = 0.0;
  load_tile(0);
#pragma unroll 1
  for (int t = 0; t < TPW; ++t) {
    const int64_t r0 = tile_row0(t);
    if (r0 >= S) break;  // uniform: later tiles of this wave start later still
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      *reinterpret_cast<uint4 *>(my + (i * RPL + lr) * LSTR + lc * 16) = buf[i];
    // the wave's LDS operations complete in order: the reads below see the
    // writes above, and the next tile's writes follow these reads
    asm volatile("" ::: "memory");
    uint4 a[NC][NP];
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int p = 0; p < NP; ++p)
        a[c][p] = *reinterpret_cast<const uint4 *>(my + (16 * c + (lane & 15)) * LSTR + p * 64 +
                                                   kq * 16);
    asm volatile("" ::: "memory");
    if (t + 1 < TPW && tile_row0(t + 1) < S) load_tile(t + 1);

    auto elem = [&](const uint4 *pc, int s) -> double {
      const uint4 v = pc[s / EPP];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
      const int e = s % EPP;
      if (BF16) return (double)((e & 1) ? bf16_hi(w[e >> 1]) : bf16_lo(w[e >> 1]));
      return (double)__uint_as_float(w[e]);
    };
    double acc[NC][2];
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[c][0] = acc[c][1] = 0.0;
#pragma unroll
    for (int s = 0; s < NH; ++s)
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          acc[c][hh] = __builtin_amdgcn_mfma_f64_4x4x4f64(elem(a[c], s + hh * NH),
                                                          bql[(s + hh * NH) * 16], acc[c][hh],
                                                          0, 0, 0);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int64_t s = r0 + 16 * c + zrow;
      if (g < G && s < S) {
        const double z = (acc[c][0] + acc[c][1]) * scale;
        zspill[(bh * S_pad + s) * G + g] = z;
        // one exp per score: exp(-|z - m|) either rescales the old sum or is
        // the new term
        const double dz = z - m_l;
        const double e = exp(-fabs(dz));
        const bool up = dz > 0.0;
        l_l = up ? fma(l_l, e, 1.0) : l_l + e;
        m_l = up ? z : m_l;
      }
    }
  }

  // chunk statistics of head g: max over the 16 lanes of g in each wave and
  // over the waves, then the rescaled sums in the same order
  double m = m_l;
#pragma unroll
  for (int off = 4; off <= 32; off <<= 1) m = fmax(m, __shfl_xor(m, off, 64));
  if (lane < 4) red[wave][lane] = m;
  __syncthreads();
  const double mc = fmax(fmax(red[0][g], red[1][g]), fmax(red[2][g], red[3][g]));
  double v = m_l == -INFINITY ? 0.0 : l_l * exp(m_l - mc);
#pragma unroll
  for (int off = 4; off <= 32; off <<= 1) v += __shfl_xor(v, off, 64);
  if (lane < 4) red2[wave][lane] = v;
  __syncthreads();
  if (wave == 0 && lane < G) {
    double *p = part + ((bh * nslot + chunk) * G + lane) * 2;
    p[0] = mc;
    p[1] = ((red2[0][lane] + red2[1][lane]) + red2[2][lane]) + red2[3][lane];
  }
}

// ---------------------------------------------------------------- norm
template <int G>
__global__ __launch_bounds__(256) void norm_kernel(const int32_t *__restrict__ lens,
                                                   const double *__restrict__ zspill,
                                                   const double *__restrict__ part,
                                                   uint64_t *__restrict__ keys,
                                                   uint32_t *__restrict__ hist, int Hkv,
                                                   int64_t S_pad, int nslot, int64_t max_len) {
  __shared__ uint32_t sh_hist[kHistBins];
  __shared__ double sm[G], sinv[G];
  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  const int nch = (int)((S + kScoreChunk - 1) / kScoreChunk);
  const int64_t bh = (int64_t)b * Hkv + h;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int t = threadIdx.x; t < kHistBins; t += 256) sh_hist[t] = 0u;

  // Every workgroup of this (b, h) merges the same partials in the same
  // order, so all of them see bit-identical (m_g, l_g).
  for (int g = wave; g < G; g += 4) {
    double m, inv;
    merged_stats(part, bh, nslot, nch, G, g, lane, m, inv);
    if (lane == 0) { sm[g] = m; sinv[g] = inv; }
  }
  __syncthreads();
  double m[G], inv[G];
#pragma unroll
  for (int g = 0; g < G; ++g) { m[g] = sm[g]; inv[g] = sinv[g]; }

  for (int i = 0; i < kScoreChunk / 256; ++i) {
    const int64_t s = c0 + i * 256 + threadIdx.x;
    if (c0 + i * 256 >= S) break;  // uniform
    const bool valid = s < S;
    uint64_t key = 0;
    if (valid) {
      const double *zz = zspill + (bh * S_pad + s) * G;
      double acc = 0.0;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += exp(zz[g] - m[g]) * inv[g];
      key = (uint64_t)__double_as_longlong(acc);
      keys[bh * S_pad + s] = key;
    }
    // wave-aggregated histogram update: few distinct exponents per wave
    const uint32_t bin = (uint32_t)(key >> 52) & (kHistBins - 1);
    uint64_t pending = __ballot(valid);
    while (pending) {
      const int leader = __ffsll((unsigned long long)pending) - 1;
      const uint32_t lb = __shfl(bin, leader, 64);
      const uint64_t same = __ballot(valid && bin == lb) & pending;
      if (lane == leader) atomicAdd(&sh_hist[lb], (uint32_t)__popcll(same));
      pending &= ~same;
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kHistBins; t += 256)
    if (sh_hist[t]) atomicAdd(&hist[bh * kHistBins + t], sh_hist[t]);
}

// ---------------------------------------------------------------- x query rows
// The x rows centred in the block, c0 = (block - x) / 2 ..., converted exactly
// to fp64: qx[b][h][e][v] with score row v = i * G + g for window row c0 + i
// and query head h * G + g. Clears the first-level histogram.
template <bool BF16>
__global__ __launch_bounds__(256) void rows_kernel(const void *__restrict__ q_sel,
                                                   double *__restrict__ qx,
                                                   uint32_t *__restrict__ hist,
                                                   double *__restrict__ part, int nslot,
                                                   int block, int x, int Hq, int Hkv, int D) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int G = Hq / Hkv, V = x * G, c0 = (block - x) / 2;
  const int64_t bh = (int64_t)b * Hkv + h;
  for (int t = blockIdx.z * 256 + threadIdx.x; t < D * V; t += gridDim.z * 256) {
    const int e = t / V, v = t % V, i = v / G, g = v % G;
    const int64_t src = (((int64_t)b * block + c0 + i) * Hq + h * G + g) * D + e;
    const float f = BF16 ? bf16_lo(reinterpret_cast<const uint16_t *>(q_sel)[src])
                         : reinterpret_cast<const float *>(q_sel)[src];
    qx[(bh * D + e) * V + v] = (double)f;
  }
  if (blockIdx.z == 0) {
    for (int i = threadIdx.x; i < kHistBins; i += 256) hist[bh * kHistBins + i] = 0u;
    for (int v = threadIdx.x; v < V; v += 256) {  // no tail unless tail_kernel runs
      double *p = part + ((bh * nslot + nslot - 1) * V + v) * 2;
      p[0] = -INFINITY;
      p[1] = 0.0;
    }
  }
}

// Softmax statistics of a normalisation tail: block n's draft KV, which
// block n+1's selection appends (sec. IV-B.2, steps 7-8). For every score row
// v, (max, sum of exp) of its scores over the n_tail tail rows (one lane
// each, n_tail <= 64) go to the last partial slot, which norm merges after the
// chunks; the tail rows are never ranked. tail: [b][n_tail][Hkv][D].
template <bool BF16>
__global__ __launch_bounds__(256) void tail_kernel(const double *__restrict__ qbar,
                                                   const void *__restrict__ tail, int n_tail,
                                                   double *__restrict__ part, int nslot,
                                                   int Hkv, int V, int D, double scale) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int v = wave; v < V; v += 4) {
    double z = -INFINITY;
    if (lane < n_tail) {
      const int64_t row = (((int64_t)b * n_tail + lane) * Hkv + h) * D;
      double acc = 0.0;
      for (int e = 0; e < D; ++e) {
        const double kx = BF16 ? (double)bf16_lo(reinterpret_cast<const uint16_t *>(tail)[row + e])
                               : (double)reinterpret_cast<const float *>(tail)[row + e];
        acc = fma(qbar[(bh * D + e) * V + v], kx, acc);
      }
      z = acc * scale;
    }
    double m = z;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
    double l = lane < n_tail ? exp(z - m) : 0.0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off, 64);
    if (lane == 0) {
      double *p = part + ((bh * nslot + nslot - 1) * V + v) * 2;
      p[0] = m;
      p[1] = l;
    }
  }
}

// Scores of V > 4 score rows per KV head on the fp64 matrix cores. In one
// v_mfma_f64_4x4x4_4b the four blocks hold four different groups of 4 cached
// rows (B) against the same 4 score rows (A, the same in every block), so one
// instruction forms 4 score rows x 16 cached rows: lane l of B holds cached
// row l % 16 at element slot l / 16, lane l of A holds score row l % 4 at
// slot l / 16, and the result of lane l is score row l / 16 of cached row
// l % 16. The head dimension is enumerated in the same permuted order on both
// operands, so a lane reads whole 16-byte pieces of its cached row. A
// workgroup takes NQ = 4 NG score rows (zero past V; their queries staged in
// LDS in operand order) and one chunk of 2048 cached rows; its 4 waves take
// interleaved 16-row tiles with the next tile's loads in flight. Each cached
// element is loaded and converted once per workgroup and feeds NG MFMAs (one
// per group of 4 score rows). The score-row groups of one chunk have
// consecutive linear ids, so they read the chunk at about the same time.
template <int D, bool BF16, bool PAGED, int NG>
__global__ __launch_bounds__(256, 2) void score_rows_kernel(KvView kv,
                                                            const double *__restrict__ qx,
                                                            double *__restrict__ zspill,
                                                            double *__restrict__ part,
                                                            int Hkv, int V, int nvg,
                                                            int64_t S_pad, int nslot,
                                                            double scale) {
  constexpr int ELT = BF16 ? 2 : 4;
  constexpr int EPP = 16 / ELT;                 // elements per 16-byte piece
  constexpr int NP = D * ELT / 64;              // pieces per lane and cached row
  constexpr int NS = D / 4;                     // MFMA steps over the head dimension
  constexpr int NW = 4;                         // waves per workgroup
  constexpr int TR = 16;                        // cached rows per wave tile
  constexpr int TPW = kScoreChunk / (TR * NW);  // tiles per wave
  constexpr int NQ = 4 * NG;                    // score rows per workgroup
  static_assert(NP * EPP == NS, "head dimension split");
  // queries in A-operand order: [step][slot][group][row of the group]
  __shared__ double qs[NS * 4 * NG * 4];
  __shared__ double red[NW][NQ], red2[NW][NQ];

  // score-row group fastest, then (KV head, sequence), then chunk (see
  // chunk_major)
  const int64_t nbh = (int64_t)gridDim.y * gridDim.z;
  const int64_t lin =
      blockIdx.x + (int64_t)gridDim.x * (blockIdx.y + (int64_t)gridDim.y * blockIdx.z);
  const int vg = (int)(lin % nvg);
  const int64_t rest = lin / nvg;
  const int chunk = (int)(rest / nbh), bhi = (int)(rest - (int64_t)chunk * nbh);
  const int h = bhi % (int)gridDim.y, b = bhi / (int)gridDim.y;
  const int64_t S = kv_len(kv, b);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int kq = lane >> 4;   // element slot (A and B); score row of the result
  const int cr = lane & 15;   // cached row of B and of the result
  const int ia = lane & 3;    // score row of A

  for (int t = threadIdx.x; t < NS * 4 * NG * 4; t += 256) {
    const int i = t % 4, g = (t / 4) % NG, k = (t / (4 * NG)) % 4, st = t / (16 * NG);
    const int e = (st / EPP) * (4 * EPP) + k * EPP + st % EPP;
    const int v = vg * NQ + 4 * g + i;
    qs[t] = v < V ? qx[(bh * D + e) * V + v] : 0.0;
  }
  __shared__ int32_t spt[PAGED ? kChunkPages : 1];
  if constexpr (PAGED) stage_chunk_pages(kv, b, c0, S, spt);
  __syncthreads();

  const char *kbase = kv.k + ((int64_t)b * kv.sb + (int64_t)h * kv.sh) * ELT + kq * 16;
  // 16-byte piece p of cached row s (the lane's slot)
  auto row_ptr = [&](int64_t s) -> const char * {
    if (PAGED) {
      const int64_t page = spt[(s >> kv.page_shift) - (c0 >> kv.page_shift)];
      return kv.k + (page * kv.sp + (int64_t)h * kv.sh +
                     (s & ((1 << kv.page_shift) - 1)) * kv.ss) * ELT + kq * 16;
    }
    return kbase + s * kv.ss * ELT;
  };
  auto tile_row0 = [&](int t) { return c0 + (int64_t)(t * NW + wave) * TR; };
  uint4 kb[2][NP];
  auto load_tile = [&](int t, uint4 (&dst)[NP]) {
    const int64_t r0 = tile_row0(t);
    const int64_t s = r0 + cr;
    const bool ok = s < S;
    const char *p = row_ptr(ok ? s : r0);
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      dst[q] = make_uint4(0u, 0u, 0u, 0u);
      if (ok) dst[q] = ldg16_nt(p + q * 64);
    }
  };
  auto elem = [&](const uint4 *pc, int s) -> double {
    const uint4 v = pc[s / EPP];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    const int e = s % EPP;
    if (BF16) return (double)((e & 1) ? bf16_hi(w[e >> 1]) : bf16_lo(w[e >> 1]));
    return (double)__uint_as_float(w[e]);
  };

  double m_l[NG], l_l[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) { m_l[g] = -INFINITY; l_l[g] = 0.0; }
  const double *qa = qs + kq * (4 * NG) + ia;
  auto step = [&](int t, uint4 (&cur)[NP], uint4 (&nxt)[NP]) -> bool {
    const int64_t r0 = tile_row0(t);
    if (r0 >= S) return false;  // uniform: later tiles of this wave start later still
    if (t + 1 < TPW && tile_row0(t + 1) < S) load_tile(t + 1, nxt);
    double acc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[g] = 0.0;
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const double bk = elem(cur, st);
#pragma unroll
      for (int g = 0; g < NG; ++g)
        acc[g] = __builtin_amdgcn_mfma_f64_4x4x4f64(qa[st * (16 * NG) + 4 * g], bk, acc[g], 0,
                                                    0, 0);
    }
    const int64_t s = r0 + cr;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int v = vg * NQ + 4 * g + kq;
      if (v < V && s < S) {
        const double z = acc[g] * scale;
        zspill[(bh * S_pad + s) * V + v] = z;
        // one exp per score: exp(-|z - m|) either rescales the old sum or is
        // the new term
        const double dz = z - m_l[g];
        const double e = exp(-fabs(dz));
        const bool up = dz > 0.0;
        l_l[g] = up ? fma(l_l[g], e, 1.0) : l_l[g] + e;
        m_l[g] = up ? z : m_l[g];
      }
    }
    return true;
  };
  load_tile(0, kb[0]);
#pragma unroll 1
  for (int t = 0; t < TPW; t += 2) {
    if (!step(t, kb[0], kb[1])) break;
    if (!step(t + 1, kb[1], kb[0])) break;
  }

  // chunk statistics of each score row: over its 16 cached-row lanes, then the
  // waves, in a fixed order
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    double m = m_l[g];
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) m = fmax(m, __shfl_xor(m, off, 64));
    if (cr == 0) red[wave][4 * g + kq] = m;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int slot = 4 * g + kq;
    const double mc = fmax(fmax(red[0][slot], red[1][slot]), fmax(red[2][slot], red[3][slot]));
    double v = m_l[g] == -INFINITY ? 0.0 : l_l[g] * exp(m_l[g] - mc);
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off, 64);
    if (cr == 0) red2[wave][slot] = v;
  }
  __syncthreads();
  for (int slot = threadIdx.x; slot < NQ; slot += 256) {
    const int v = vg * NQ + slot;
    if (v >= V) continue;
    const double mc = fmax(fmax(red[0][slot], red[1][slot]), fmax(red[2][slot], red[3][slot]));
    double *p = part + ((bh * nslot + chunk) * V + v) * 2;
    p[0] = mc;
    p[1] = ((red2[0][slot] + red2[1][slot]) + red2[2][slot]) + red2[3][slot];
  }
}

// GQA importance for any number V of score rows per KV head: as norm_kernel,
// with the statistics in LDS and LPR lanes per cached row (the power of two
// that gives each lane at most 8 of the V terms, up to 64 lanes) summing the
// terms, combined by a butterfly of shuffles (every lane of the row ends with
// the same sum, so equal score rows give equal keys).
__global__ __launch_bounds__(256) void norm_rows_kernel(const int32_t *__restrict__ lens,
                                                        const double *__restrict__ zspill,
                                                        const double *__restrict__ part,
                                                        uint64_t *__restrict__ keys,
                                                        uint32_t *__restrict__ hist, int Hkv,
                                                        int V, int64_t S_pad, int nslot,
                                                        int64_t max_len) {
  __shared__ uint32_t sh_hist[kHistBins];
  __shared__ double sm[kMaxScoreRows], sinv[kMaxScoreRows];
  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  const int nch = (int)((S + kScoreChunk - 1) / kScoreChunk);
  const int64_t bh = (int64_t)b * Hkv + h;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int t = threadIdx.x; t < kHistBins; t += 256) sh_hist[t] = 0u;

  // every workgroup of this (b, h) merges the same partials in the same order
  for (int v = wave; v < V; v += 4) {
    double m, inv;
    merged_stats(part, bh, nslot, nch, V, v, lane, m, inv);
    if (lane == 0) { sm[v] = m; sinv[v] = inv; }
  }
  __syncthreads();

  int lpr = 1;
  while (lpr * 8 < V && lpr < 64) lpr <<= 1;
  const int rpi = 64 / lpr;                 // cached rows per wave and round
  const int sub = lane / lpr, q = lane % lpr;
  const int64_t c1 = min(c0 + (int64_t)kScoreChunk, S);
  for (int64_t base = c0 + (int64_t)wave * rpi; base < c1; base += 4 * rpi) {
    const int64_t s = base + sub;
    const bool valid = s < c1;
    double acc = 0.0;
    if (valid) {
      const double *zz = zspill + (bh * S_pad + s) * V;
      for (int v0 = q; v0 < V; v0 += 8 * lpr) {
        // up to 8 terms of this lane, every load issued before the exps
        double z[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) z[u] = v0 + u * lpr < V ? zz[v0 + u * lpr] : 0.0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int v = v0 + u * lpr;
          if (v < V) acc += exp(z[u] - sm[v]) * sinv[v];
        }
      }
    }
    for (int off = lpr >> 1; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
    const bool lead = valid && q == 0;
    uint64_t key = 0;
    if (lead) {
      key = (uint64_t)__double_as_longlong(acc);
      keys[bh * S_pad + s] = key;
    }
    const uint32_t bin = (uint32_t)(key >> 52) & (kHistBins - 1);
    uint64_t pending = __ballot(lead);
    while (pending) {
      const int leader = __ffsll((unsigned long long)pending) - 1;
      const uint32_t lb = __shfl(bin, leader, 64);
      const uint64_t same = __ballot(lead && bin == lb) & pending;
      if (lane == leader) atomicAdd(&sh_hist[lb], (uint32_t)__popcll(same));
      pending &= ~same;
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kHistBins; t += 256)
    if (sh_hist[t]) atomicAdd(&hist[bh * kHistBins + t], sh_hist[t]);
}

// ---------------------------------------------------------------- attention output
// Optional output of the selection: the attention of every score row v over
// the cache and the tail, o_v = sum_s exp(z_v[s] - m_v) / l_v * v_s (the
// output accumulator that the paper's fused kernel keeps beside (m, l),
// sec. IV-B.4), from the spilled fp64 scores and the merged statistics, with
// fp32 weights and fp32 accumulation. out_kernel: one workgroup per (chunk,
// KV head, sequence) writes the chunk's partial sum [V][D]. A cached row is
// read as D / EPL 16-byte pieces by as many consecutive threads (its row
// slot); each thread keeps NV score rows x EPL elements of one piece position
// and loads the pieces of a 128-row tile all at once; the weights of the tile
// are formed once in LDS. At the end the row slots are summed in a fixed
// order: shuffles within a wave, then the four waves through LDS.
template <int D, int NV, bool BF16>
__global__ __launch_bounds__(256) void out_kernel(KvView kv, const double *__restrict__ zspill,
                                                  const double *__restrict__ part,
                                                  float *__restrict__ opart, int Hkv, int V,
                                                  int64_t S_pad, int nslot) {
  constexpr int ELT = BF16 ? 2 : 4;
  constexpr int EPL = 16 / ELT;   // elements per 16-byte piece
  constexpr int SEG = D / EPL;    // pieces per cached row
  constexpr int RS = 256 / SEG;   // cached rows per step (row slots)
  constexpr int WRS = 64 / SEG;   // row slots per wave
  constexpr int TR = 128;         // cached rows per weight tile
  constexpr int SPT = TR / RS;    // steps per tile
  __shared__ double sm[kMaxScoreRows], sinv[kMaxScoreRows];
  __shared__ float wt[TR][NV];
  __shared__ float red[4][NV][D];
  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t S = kv_len(kv, b);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S) return;
  const int nch = (int)((S + kScoreChunk - 1) / kScoreChunk);
  const int64_t bh = (int64_t)b * Hkv + h;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int v = wave; v < V; v += 4) {
    double m, inv;
    merged_stats(part, bh, nslot, nch, V, v, lane, m, inv);
    if (lane == 0) { sm[v] = m; sinv[v] = inv; }
  }
  __syncthreads();
  const int seg = threadIdx.x % SEG, rslot = threadIdx.x / SEG;
  const int64_t c1 = min(c0 + (int64_t)kScoreChunk, S);
  for (int vb0 = 0; vb0 < V; vb0 += NV) {
    float acc[NV][EPL];
#pragma unroll
    for (int j = 0; j < NV; ++j)
#pragma unroll
      for (int u = 0; u < EPL; ++u) acc[j][u] = 0.f;
    for (int64_t r0 = c0; r0 < c1; r0 += TR) {
      for (int i = threadIdx.x; i < TR * NV; i += 256) {
        const int rr = i / NV, v = vb0 + i % NV;
        const int64_t s = r0 + rr;
        float w = 0.f;
        if (s < c1 && v < V)
          w = (float)(exp(zspill[(bh * S_pad + s) * V + v] - sm[v]) * sinv[v]);
        wt[rr][i % NV] = w;
      }
      __syncthreads();
      uint4 pc[SPT];
#pragma unroll
      for (int st = 0; st < SPT; ++st) {
        const int64_t s = r0 + st * RS + rslot;
        pc[st] = make_uint4(0u, 0u, 0u, 0u);
        if (s < c1) pc[st] = ldg16(kv.v + kv_row(kv, b, h, s) * ELT + seg * 16);
      }
#pragma unroll
      for (int st = 0; st < SPT; ++st) {
        const int rr = st * RS + rslot;
        const uint32_t w4[4] = {pc[st].x, pc[st].y, pc[st].z, pc[st].w};
        float x[EPL];
#pragma unroll
        for (int u = 0; u < EPL; ++u)
          x[u] = BF16 ? ((u & 1) ? bf16_hi(w4[u >> 1]) : bf16_lo(w4[u >> 1]))
                      : __uint_as_float(w4[u]);
#pragma unroll
        for (int j = 0; j < NV; ++j) {
          const float w = wt[rr][j];
#pragma unroll
          for (int u = 0; u < EPL; ++u) acc[j][u] = fmaf(w, x[u], acc[j][u]);
        }
      }
      __syncthreads();
    }
    // row slots of a wave (lanes seg + SEG r) in a fixed tree, then the waves
#pragma unroll
    for (int off = SEG; off < 64; off <<= 1)
#pragma unroll
      for (int j = 0; j < NV; ++j)
#pragma unroll
        for (int u = 0; u < EPL; ++u) acc[j][u] += __shfl_xor(acc[j][u], off, 64);
    static_assert(WRS >= 1, "a wave holds at least one row slot");
    if (lane < SEG)
#pragma unroll
      for (int j = 0; j < NV; ++j)
#pragma unroll
        for (int u = 0; u < EPL; ++u) red[wave][j][seg * EPL + u] = acc[j][u];
    __syncthreads();
    for (int i = threadIdx.x; i < NV * D; i += 256) {
      const int j = i / D, e = i % D, v = vb0 + j;
      if (v < V)
        opart[((bh * nslot + chunk) * V + v) * D + e] =
            ((red[0][j][e] + red[1][j][e]) + red[2][j][e]) + red[3][j][e];
    }
    __syncthreads();
  }
}

// The tail rows' part of the attention output, into the last partial slot:
// one wave per score row; the lanes first form the tail scores (as
// tail_kernel does) and weights, then sum weight x V over the tail rows for
// two elements each.
template <bool BF16>
__global__ __launch_bounds__(256) void out_tail_kernel(const double *__restrict__ qbar,
                                                       const void *__restrict__ tail_k,
                                                       const void *__restrict__ tail_v,
                                                       int n_tail, const int32_t *lens,
                                                       int64_t max_len,
                                                       const double *__restrict__ part,
                                                       float *__restrict__ opart, int Hkv, int V,
                                                       int D, int nslot, double scale) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int nch = (int)((S + kScoreChunk - 1) / kScoreChunk);
  auto elem = [&](const void *p, int64_t i) -> double {
    return BF16 ? (double)bf16_lo(reinterpret_cast<const uint16_t *>(p)[i])
                : (double)reinterpret_cast<const float *>(p)[i];
  };
  for (int v = wave; v < V; v += 4) {
    double m, inv;
    merged_stats(part, bh, nslot, nch, V, v, lane, m, inv);
    float w = 0.f;
    if (lane < n_tail) {
      const int64_t row = (((int64_t)b * n_tail + lane) * Hkv + h) * D;
      double acc = 0.0;
      for (int e = 0; e < D; ++e) acc = fma(qbar[(bh * D + e) * V + v], elem(tail_k, row + e), acc);
      w = (float)(exp(acc * scale - m) * inv);
    }
    for (int e = lane; e < D; e += 64) {
      float o = 0.f;
      for (int t = 0; t < n_tail; ++t) {
        const float wt = __shfl(w, t, 64);
        o = fmaf(wt, (float)elem(tail_v, (((int64_t)b * n_tail + t) * Hkv + h) * D + e), o);
      }
      opart[((bh * nslot + nslot - 1) * V + v) * D + e] = o;
    }
  }
}

// o[b][i][h G + g][e] (v = i G + g) = the chunks' parts in chunk order, then
// the tail's; bf16 outputs rounded to nearest-even.
template <bool BF16>
__global__ __launch_bounds__(256) void out_combine_kernel(const int32_t *lens, int64_t max_len,
                                                          const float *__restrict__ opart,
                                                          void *__restrict__ o_out, int n_tail,
                                                          int Hq, int Hkv, int V, int D,
                                                          int nslot) {
  const int h = blockIdx.y, b = blockIdx.z;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= V * D) return;
  const int v = t / D, e = t % D, G = Hq / Hkv, i = v / G, g = v % G;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int nch = (int)((S + kScoreChunk - 1) / kScoreChunk);
  float acc = 0.f;
  for (int c = 0; c < nch; ++c) acc += opart[((bh * nslot + c) * V + v) * D + e];
  if (n_tail > 0) acc += opart[((bh * nslot + nslot - 1) * V + v) * D + e];
  const int64_t dst = (((int64_t)b * (V / G) + i) * Hq + h * G + g) * D + e;
  if (BF16)
    reinterpret_cast<uint16_t *>(o_out)[dst] = (uint16_t)f32_to_bf16_rne(acc);
  else
    reinterpret_cast<float *>(o_out)[dst] = acc;
}

// ---------------------------------------------------------------- topk
// Block-wide exclusive scan of one int per thread (1024 threads).
__device__ __forceinline__ int block_excl_scan(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kTopkThreads / 64; ++w) {
    const int x = wsum[w];
    before += (w < wave) ? x : 0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return before + incl - v;
}

// All threads: the digit d with above(d) < r <= above(d) + cnt[d], where
// above(d) counts keys in bins > d. Thread t sums the bins at ranks
// [per t, per (t + 1)) from the top; a block scan of those sums locates the
// one thread whose bins hold rank r. Results go to shared memory.
__device__ __forceinline__ void find_digit(const uint32_t *cnt, int nbins, int r, int *wsum,
                                           int *s_digit, int *s_above, int *s_cnt) {
  const int tid = threadIdx.x;
  const int per = nbins > kTopkThreads ? nbins / kTopkThreads : 1;  // nbins: power of two
  const int hi = nbins - per * tid;                                 // bins [hi - per, hi)
  int mine = 0;
  for (int i = 0; i < per; ++i) {
    const int bin = hi - 1 - i;
    if (bin >= 0) mine += (int)cnt[bin];
  }
  int total;
  const int before = block_excl_scan(mine, wsum, &total);
  if (before < r && r <= before + mine) {
    int acc = before;
    for (int i = 0; i < per; ++i) {
      const int bin = hi - 1 - i;
      if (bin < 0) break;
      const int c = (int)cnt[bin];
      if (acc + c >= r) { *s_digit = bin; *s_above = acc; *s_cnt = c; break; }
      acc += c;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(
    const int32_t *__restrict__ lens, const int32_t *__restrict__ kps, int k_max,
    const uint64_t *__restrict__ keys, const uint32_t *__restrict__ hist,
    int32_t *__restrict__ idx_out, uint64_t *__restrict__ cut, int Hkv, int64_t S_pad,
    int64_t max_len) {
  constexpr int KPT = kKeysPerThread;
  __shared__ uint32_t cnt[kHistBins];
  __shared__ uint64_t cand[kCandCap];
  __shared__ int wsum[kTopkThreads / 64];
  __shared__ int s_digit, s_above, s_cnt, s_ncand;

  const int h = blockIdx.x, b = blockIdx.y;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int k = clamp_k(kps[b], S, k_max);
  int32_t *out = idx_out + bh * k_max;
  const uint64_t *kb = keys + bh * S_pad;
  const uint64_t lanes_below = (1ull << lane) - 1ull;

  if (k == 0 || k == S) {
    for (int j = tid; j < k_max; j += kTopkThreads) out[j] = j < k ? j : -1;
    if (tid == 0) cut[bh * 4 + 3] = 0;  // nothing left for the emission kernels
    return;
  }

  for (int i = tid; i < kHistBins; i += kTopkThreads) cnt[i] = hist[bh * kHistBins + i];
  if (tid == 0) s_ncand = 0;
  __syncthreads();
  find_digit(cnt, kHistBins, k, wsum, &s_digit, &s_above, &s_cnt);
  uint64_t P = (uint64_t)s_digit;
  int r = k - s_above;
  int c = s_cnt;
  int L = 52;
  bool in_lds = false;
  int ncand = 0;

  // compact the keys whose top (64 - L) bits equal P into LDS: KPT keys per
  // thread in flight, one slot reservation per wave and round
  auto compact = [&]() {
    for (int64_t base = 0; base < S; base += (int64_t)kTopkThreads * KPT) {
      uint64_t key[KPT];
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int64_t s = base + (int64_t)u * kTopkThreads + tid;
        key[u] = s < S ? kb[s] : 0;
      }
      uint64_t bal[KPT];
      int n = 0;
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int64_t s = base + (int64_t)u * kTopkThreads + tid;
        bal[u] = __ballot(s < S && (key[u] >> L) == P);
        n += __popcll(bal[u]);
      }
      int slot = 0;
      if (lane == 0 && n) slot = atomicAdd(&s_ncand, n);
      slot = __shfl(slot, 0, 64);
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        if ((bal[u] >> lane) & 1ull) {
          const int at = slot + __popcll(bal[u] & lanes_below);
          if (at < kCandCap) cand[at] = key[u];
        }
        slot += __popcll(bal[u]);
      }
    }
    __syncthreads();
    ncand = min(s_ncand, kCandCap);
    in_lds = true;
  };

  if (c != r && c <= kCandCap) compact();
  while (c != r && L > 0) {
    const int nb = L < 11 ? L : 11;
    const int L2 = L - nb;
    const uint32_t mask = (1u << nb) - 1u;
    for (int i = tid; i < (1 << nb); i += kTopkThreads) cnt[i] = 0u;
    __syncthreads();
    if (in_lds) {
      for (int i = tid; i < ncand; i += kTopkThreads) {
        const uint64_t key = cand[i];
        if ((key >> L) == P) atomicAdd(&cnt[(uint32_t)(key >> L2) & mask], 1u);
      }
    } else {
      for (int64_t base = 0; base < S; base += (int64_t)kTopkThreads * KPT) {
        uint64_t key[KPT];
#pragma unroll
        for (int u = 0; u < KPT; ++u) {
          const int64_t s = base + (int64_t)u * kTopkThreads + tid;
          key[u] = s < S ? kb[s] : ~0ull;
        }
#pragma unroll
        for (int u = 0; u < KPT; ++u)
          if (base + (int64_t)u * kTopkThreads + tid < S && (key[u] >> L) == P)
            atomicAdd(&cnt[(uint32_t)(key[u] >> L2) & mask], 1u);
      }
    }
    __syncthreads();
    find_digit(cnt, 1 << nb, r, wsum, &s_digit, &s_above, &s_cnt);
    r -= s_above;
    P = (P << nb) | (uint64_t)s_digit;
    c = s_cnt;
    L = L2;
    __syncthreads();
    if (!in_lds && c != r && c <= kCandCap) compact();
  }

  // The cut, for the ordered emission of emit_count_kernel and
  // emit_write_kernel: keys whose top (64 - L) bits exceed P are taken; keys
  // of the boundary bucket (top bits equal to P; exact ties once L == 0) all
  // of them when the bucket holds exactly r keys, else the r of lowest index.
  if (tid == 0) {
    cut[bh * 4 + 0] = P;
    cut[bh * 4 + 1] = (uint64_t)L;
    cut[bh * 4 + 2] = (uint64_t)r;
    cut[bh * 4 + 3] = (uint64_t)(c == r ? 2 : 1);  // 2: whole bucket, 1: r lowest
  }
  for (int j = k + tid; j < k_max; j += kTopkThreads) out[j] = -1;
}

// Ordered emission of the top-k, one workgroup per chunk of 2048 keys of a
// (KV head, sequence): emit_count_kernel marks and counts the chunk's keys
// above the cut and in the boundary bucket (one byte of each mask per 8
// consecutive keys); emit_write_kernel adds up the counts of the chunks
// before its own, and each thread, owning 8 consecutive keys, finds its
// output positions from the marks with one block scan, so the indices come
// out in ascending order.
__device__ __forceinline__ void chunk_marks(const uint64_t *kb, int64_t s0, int64_t S,
                                            uint64_t P, int L, uint32_t &gt, uint32_t &eq) {
  uint64_t key[8];
  if (s0 + 8 <= S) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint4 v = *reinterpret_cast<const uint4 *>(kb + s0 + 2 * j);
      key[2 * j] = (uint64_t)v.x | ((uint64_t)v.y << 32);
      key[2 * j + 1] = (uint64_t)v.z | ((uint64_t)v.w << 32);
    }
  } else {
#pragma unroll
    for (int u = 0; u < 8; ++u) key[u] = s0 + u < S ? kb[s0 + u] : 0;
  }
  gt = eq = 0;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const bool valid = s0 + u < S;
    // (L == 64 never happens: the first digit already fixes 12 bits)
    const uint64_t hi = valid ? (key[u] >> L) : 0;
    gt |= (uint32_t)(valid && hi > P) << u;
    eq |= (uint32_t)(valid && hi == P) << u;
  }
}

__global__ __launch_bounds__(256) void emit_count_kernel(
    const int32_t *__restrict__ lens, const uint64_t *__restrict__ keys,
    const uint64_t *__restrict__ cut, uint32_t *__restrict__ ecnt, uint8_t *__restrict__ emark,
    int Hkv, int64_t S_pad, int nchunk, int64_t max_len) {
  __shared__ uint32_t wsum[4];
  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  if (c0 >= S || cut[bh * 4 + 3] == 0) return;
  uint32_t gt, eq;
  chunk_marks(keys + bh * S_pad, c0 + threadIdx.x * 8, S, cut[bh * 4], (int)cut[bh * 4 + 1],
              gt, eq);
  uint8_t *mk = emark + (bh * nchunk + chunk) * 512;
  mk[threadIdx.x] = (uint8_t)gt;
  mk[256 + threadIdx.x] = (uint8_t)eq;
  uint32_t v = ((uint32_t)__popc(gt) << 16) | (uint32_t)__popc(eq);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) ecnt[bh * nchunk + chunk] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

__global__ __launch_bounds__(256) void emit_write_kernel(
    const int32_t *__restrict__ lens, const int32_t *__restrict__ kps, int k_max,
    const uint64_t *__restrict__ cut, const uint32_t *__restrict__ ecnt,
    const uint8_t *__restrict__ emark, int32_t *__restrict__ idx_out, int Hkv, int nchunk,
    int64_t max_len) {
  __shared__ uint32_t wsum[4], wbase[4];
  const ChunkOf cid = chunk_major();
  const int chunk = cid.chunk, h = cid.h, b = cid.b;
  const int64_t bh = (int64_t)b * Hkv + h;
  const int64_t S = min(max((int64_t)lens[b], (int64_t)0), max_len);
  const int64_t c0 = (int64_t)chunk * kScoreChunk;
  const uint64_t mode = cut[bh * 4 + 3];
  if (c0 >= S || mode == 0) return;
  const int k = clamp_k(kps[b], S, k_max);
  const int r = (int)cut[bh * 4 + 2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // keys above the cut and in the bucket in the chunks before this one (each
  // count below 2^16: a chunk holds 2048 keys)
  uint32_t gt_before = 0, eq_before = 0;
  for (int c = tid; c < chunk; c += 256) {
    const uint32_t v = ecnt[bh * nchunk + c];
    gt_before += v >> 16;
    eq_before += v & 0xffffu;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    gt_before += __shfl_xor(gt_before, off, 64);
    eq_before += __shfl_xor(eq_before, off, 64);
  }
  if (lane == 0) { wsum[wave] = gt_before; wbase[wave] = eq_before; }
  __syncthreads();
  gt_before = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
  eq_before = ((wbase[0] + wbase[1]) + wbase[2]) + wbase[3];
  __syncthreads();

  const int64_t s0 = c0 + tid * 8;
  const uint8_t *mk = emark + (bh * nchunk + chunk) * 512;
  const uint32_t gt = mk[tid], eq = mk[256 + tid];
  // exclusive scan over the threads of (keys above, bucket keys), packed
  const uint32_t mine = ((uint32_t)__popc(gt) << 16) | (uint32_t)__popc(eq);
  uint32_t incl = mine;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  uint32_t excl = incl - mine;
  for (int w = 0; w < wave; ++w) excl += wsum[w];
  // bucket keys before this thread's, over the whole sequence, and how many
  // of them are taken; then this thread's first output position
  const int eq_rank = (int)(eq_before + (excl & 0xffffu));
  const bool whole = mode == 2;
  auto taken_eq = [&](int n) { return whole ? n : max(0, min(n, r)); };
  int pos = (int)(gt_before + (excl >> 16)) + taken_eq(eq_rank);
  int rank = eq_rank;
  int32_t *out = idx_out + bh * k_max;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    bool take = (gt >> u) & 1u;
    if ((eq >> u) & 1u) {
      take = whole || rank < r;
      ++rank;
    }
    if (take) {
      if (pos < k) out[pos] = (int32_t)(s0 + u);  // counts are exact; guard anyway
      ++pos;
    }
  }
}

// Top-k of every (KV head, sequence) from the keys and the first-level
// histogram: the cut, then the chunk-parallel ordered emission.
void launch_topk(const KvView &kv, int batch, int Hkv, const int32_t *k_per_seq, int k_max,
                 int32_t *idx_out, const SelectWs &ws, hipStream_t stream) {
  topk_kernel<<<dim3(Hkv, batch), kTopkThreads, 0, stream>>>(
      kv.lens, k_per_seq, k_max, ws.keys, ws.hist, idx_out, ws.cut, Hkv, ws.S_pad, kv.max_len);
  const dim3 grid(ws.nchunk, Hkv, batch);
  emit_count_kernel<<<grid, 256, 0, stream>>>(kv.lens, ws.keys, ws.cut, ws.ecnt, ws.emark, Hkv,
                                              ws.S_pad, ws.nchunk, kv.max_len);
  emit_write_kernel<<<grid, 256, 0, stream>>>(kv.lens, k_per_seq, k_max, ws.cut, ws.ecnt,
                                              ws.emark, idx_out, Hkv, ws.nchunk, kv.max_len);
}

// The optional attention output (after norm has written the keys: the
// statistics are in place), o_out [b][V / G][Hq][D].
template <int D, bool BF16>
void launch_out(const KvView &kv, int batch, int Hq, int Hkv, int V, const void *tail,
                const void *tail_v, int n_tail, void *o_out, const SelectWs &ws, int nslot,
                double scale, hipStream_t stream) {
  const dim3 grid(ws.nchunk, Hkv, batch);
  if (V <= 4)
    out_kernel<D, 4, BF16><<<grid, 256, 0, stream>>>(kv, ws.espill, ws.part, ws.opart, Hkv, V,
                                                     ws.S_pad, nslot);
  else if (V <= 8)
    out_kernel<D, 8, BF16><<<grid, 256, 0, stream>>>(kv, ws.espill, ws.part, ws.opart, Hkv, V,
                                                     ws.S_pad, nslot);
  else
    out_kernel<D, 16, BF16><<<grid, 256, 0, stream>>>(kv, ws.espill, ws.part, ws.opart, Hkv, V,
                                                      ws.S_pad, nslot);
  if (n_tail > 0)
    out_tail_kernel<BF16><<<dim3(Hkv, batch), 256, 0, stream>>>(
        ws.qbar, tail, tail_v, n_tail, kv.lens, kv.max_len, ws.part, ws.opart, Hkv, V, D, nslot,
        scale);
  out_combine_kernel<BF16><<<dim3((V * D + 255) / 256, Hkv, batch), 256, 0, stream>>>(
      kv.lens, kv.max_len, ws.opart, o_out, n_tail, Hq, Hkv, V, D, nslot);
}

template <int D, int G, bool BF16>
hipError_t launch_select_t(int batch, int block, const void *q_sel, const KvView &kv,
                           int Hq, int Hkv, const void *tail, const void *tail_v, int n_tail,
                           const int32_t *k_per_seq, int k_max, int32_t *idx_out,
                           void *o_out, const SelectWs &ws, hipStream_t stream) {
  const double scale = 1.0 / sqrt((double)D);
  const int nslot = ws.nchunk + 1;  // partial slots per (b, h): chunks, then the tail
  repq_kernel<D, G, BF16><<<dim3(Hkv, batch, (D * G + 255) / 256), 256, 0, stream>>>(
      q_sel, ws.qbar, ws.hist, ws.part, nslot, block, Hq, Hkv);
  if (n_tail > 0)
    tail_kernel<BF16><<<dim3(Hkv, batch), 256, 0, stream>>>(ws.qbar, tail, n_tail, ws.part,
                                                          nslot, Hkv, G, D, scale);
  const dim3 grid(ws.nchunk, Hkv, batch);
  if constexpr (G <= 4) {
    if (kv.pt)
      score_mfma_kernel<D, G, BF16, true><<<grid, 256, 0, stream>>>(
          kv, ws.qbar, ws.espill, ws.part, Hkv, ws.S_pad, nslot, scale);
    else
      score_mfma_kernel<D, G, BF16, false><<<grid, 256, 0, stream>>>(
          kv, ws.qbar, ws.espill, ws.part, Hkv, ws.S_pad, nslot, scale);
  } else {
    if (kv.pt)
      score_kernel<D, G, BF16, true><<<grid, 256, 0, stream>>>(kv, ws.qbar, ws.espill, ws.part,
                                                               Hkv, ws.S_pad, nslot, scale);
    else
      score_kernel<D, G, BF16, false><<<grid, 256, 0, stream>>>(kv, ws.qbar, ws.espill, ws.part,
                                                                Hkv, ws.S_pad, nslot, scale);
  }
  norm_kernel<G><<<grid, 256, 0, stream>>>(kv.lens, ws.espill, ws.part, ws.keys, ws.hist,
                                           Hkv, ws.S_pad, nslot, kv.max_len);
  launch_topk(kv, batch, Hkv, k_per_seq, k_max, idx_out, ws, stream);
  if (o_out)
    launch_out<D, BF16>(kv, batch, Hq, Hkv, G, tail, tail_v, n_tail, o_out, ws, nslot, scale,
                        stream);
  return hipGetLastError();
}

template <int D, int V, bool BF16>
void launch_score_norm_small(const KvView &kv, int batch, int Hkv, const SelectWs &ws,
                             int nslot, double scale, hipStream_t stream) {
  const dim3 grid(ws.nchunk, Hkv, batch);
  if (kv.pt)
    score_mfma_kernel<D, V, BF16, true><<<grid, 256, 0, stream>>>(
        kv, ws.qbar, ws.espill, ws.part, Hkv, ws.S_pad, nslot, scale);
  else
    score_mfma_kernel<D, V, BF16, false><<<grid, 256, 0, stream>>>(
        kv, ws.qbar, ws.espill, ws.part, Hkv, ws.S_pad, nslot, scale);
  norm_kernel<V><<<grid, 256, 0, stream>>>(kv.lens, ws.espill, ws.part, ws.keys, ws.hist, Hkv,
                                           ws.S_pad, nslot, kv.max_len);
}

template <int D, bool BF16>
hipError_t launch_select_xq_t(int batch, int block, int x, const void *q_sel,
                              const KvView &kv, int Hq, int Hkv, const void *tail,
                              const void *tail_v, int n_tail, const int32_t *k_per_seq,
                              int k_max, int32_t *idx_out, void *o_out, const SelectWs &ws,
                              hipStream_t stream) {
  const int V = x * (Hq / Hkv);
  const double scale = 1.0 / sqrt((double)D);
  const int nslot = ws.nchunk + 1;
  const int zb = min((D * V + 255) / 256, 64);
  rows_kernel<BF16><<<dim3(Hkv, batch, zb), 256, 0, stream>>>(q_sel, ws.qbar, ws.hist, ws.part,
                                                             nslot, block, x, Hq, Hkv, D);
  if (n_tail > 0)
    tail_kernel<BF16><<<dim3(Hkv, batch), 256, 0, stream>>>(ws.qbar, tail, n_tail, ws.part,
                                                          nslot, Hkv, V, D, scale);
  if (V == 1) launch_score_norm_small<D, 1, BF16>(kv, batch, Hkv, ws, nslot, scale, stream);
  else if (V == 2) launch_score_norm_small<D, 2, BF16>(kv, batch, Hkv, ws, nslot, scale, stream);
  else if (V == 4) launch_score_norm_small<D, 4, BF16>(kv, batch, Hkv, ws, nslot, scale, stream);
  else {
    // groups of 4 score rows per workgroup: the fewest that cover V, at most 16
    const int ng = V <= 8 ? 2 : V <= 16 ? 4 : V <= 32 ? 8 : 16;
    const int nvg = (V + 4 * ng - 1) / (4 * ng);
    const dim3 grid_s(ws.nchunk * nvg, Hkv, batch);
#define HERALD_SCORE_ROWS(NG_)                                                                 \
  if (ng == NG_) {                                                                             \
    if (kv.pt)                                                                                 \
      score_rows_kernel<D, BF16, true, NG_><<<grid_s, 256, 0, stream>>>(                       \
          kv, ws.qbar, ws.espill, ws.part, Hkv, V, nvg, ws.S_pad, nslot, scale);               \
    else                                                                                       \
      score_rows_kernel<D, BF16, false, NG_><<<grid_s, 256, 0, stream>>>(                      \
          kv, ws.qbar, ws.espill, ws.part, Hkv, V, nvg, ws.S_pad, nslot, scale);               \
  }
    HERALD_SCORE_ROWS(2) HERALD_SCORE_ROWS(4) HERALD_SCORE_ROWS(8) HERALD_SCORE_ROWS(16)
#undef HERALD_SCORE_ROWS
    norm_rows_kernel<<<dim3(ws.nchunk, Hkv, batch), 256, 0, stream>>>(
        kv.lens, ws.espill, ws.part, ws.keys, ws.hist, Hkv, V, ws.S_pad, nslot, kv.max_len);
  }
  launch_topk(kv, batch, Hkv, k_per_seq, k_max, idx_out, ws, stream);
  if (o_out)
    launch_out<D, BF16>(kv, batch, Hq, Hkv, V, tail, tail_v, n_tail, o_out, ws, nslot, scale,
                        stream);
  return hipGetLastError();
}

}  // namespace

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t select_ws_bytes(int batch, int Hq, int Hkv, int d, int64_t max_seq_len,
                       SelectWs *layout, char *base) {
  const int G = Hq / Hkv;
  const int nchunk = (int)((max_seq_len + kScoreChunk - 1) / kScoreChunk);
  const int64_t S_pad = (int64_t)nchunk * kScoreChunk;
  const size_t bh = (size_t)batch * Hkv;
  size_t off = 0;
  const size_t o_qbar = off; off = align256(off + bh * d * G * sizeof(double));
  const size_t o_z = off;    off = align256(off + bh * S_pad * G * sizeof(double));
  const size_t o_part = off; off = align256(off + bh * (nchunk + 1) * G * 2 * sizeof(double));
  const size_t o_keys = off; off = align256(off + bh * S_pad * sizeof(uint64_t));
  const size_t o_hist = off; off = align256(off + bh * kHistBins * sizeof(uint32_t));
  const size_t o_opart = off; off = align256(off + bh * (nchunk + 1) * G * d * sizeof(float));
  const size_t o_cut = off;  off = align256(off + bh * 4 * sizeof(uint64_t));
  const size_t o_ecnt = off; off = align256(off + bh * nchunk * sizeof(uint32_t));
  const size_t o_emark = off; off = align256(off + bh * nchunk * 2 * 256);
  if (layout) {
    layout->qbar = reinterpret_cast<double *>(base + o_qbar);
    layout->espill = reinterpret_cast<double *>(base + o_z);
    layout->part = reinterpret_cast<double *>(base + o_part);
    layout->keys = reinterpret_cast<uint64_t *>(base + o_keys);
    layout->hist = reinterpret_cast<uint32_t *>(base + o_hist);
    layout->opart = reinterpret_cast<float *>(base + o_opart);
    layout->cut = reinterpret_cast<uint64_t *>(base + o_cut);
    layout->ecnt = reinterpret_cast<uint32_t *>(base + o_ecnt);
    layout->emark = reinterpret_cast<uint8_t *>(base + o_emark);
    layout->S_pad = S_pad;
    layout->nchunk = nchunk;
  }
  return off;
}

hipError_t launch_select_xq(const herald_heads &hd, int batch, int block, int x,
                            const void *q_sel, const KvView &kv, const void *tail,
                            const void *tail_v, int n_tail, const int32_t *k_per_seq, int k_max,
                            int32_t *idx_out, void *o_out, const SelectWs &ws,
                            hipStream_t stream) {
  const bool bf = hd.dtype == HERALD_BF16;
  const int Hq = hd.num_q_heads, Hkv = hd.num_kv_heads;
#define HERALD_SELX(D_, BF_)                                                              \
  if (hd.head_dim == D_ && bf == BF_)                                                     \
    return launch_select_xq_t<D_, BF_>(batch, block, x, q_sel, kv, Hq, Hkv, tail, tail_v, \
                                       n_tail, k_per_seq, k_max, idx_out, o_out, ws, stream);
  HERALD_SELX(64, true) HERALD_SELX(64, false) HERALD_SELX(128, true) HERALD_SELX(128, false)
#undef HERALD_SELX
  return hipErrorInvalidValue;
}

hipError_t launch_select(const herald_heads &hd, int batch, int block, const void *q_sel,
                         const KvView &kv, const void *tail, const void *tail_v, int n_tail,
                         const int32_t *k_per_seq, int k_max, int32_t *idx_out, void *o_out,
                         const SelectWs &ws, hipStream_t stream) {
  const int G = hd.num_q_heads / hd.num_kv_heads;
  const bool bf = hd.dtype == HERALD_BF16;
  const int Hq = hd.num_q_heads, Hkv = hd.num_kv_heads;
#define HERALD_SEL(D_, G_)                                                              \
  if (hd.head_dim == D_ && G == G_)                                                     \
    return bf ? launch_select_t<D_, G_, true>(batch, block, q_sel, kv, Hq, Hkv, tail,   \
                                              tail_v, n_tail, k_per_seq, k_max, idx_out, \
                                              o_out, ws, stream)                         \
              : launch_select_t<D_, G_, false>(batch, block, q_sel, kv, Hq, Hkv, tail,  \
                                               tail_v, n_tail, k_per_seq, k_max,         \
                                               idx_out, o_out, ws, stream);
  HERALD_SEL(64, 1) HERALD_SEL(64, 2) HERALD_SEL(64, 4) HERALD_SEL(64, 8)
  HERALD_SEL(128, 1) HERALD_SEL(128, 2) HERALD_SEL(128, 4) HERALD_SEL(128, 8)
#undef HERALD_SEL
  return hipErrorInvalidValue;
}

}  // namespace herald
