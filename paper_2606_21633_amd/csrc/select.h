// Selection launchers and their workspace layout (host side, defined in
// select.hip).
#pragma once

#include "common.h"

namespace herald {

struct SelectWs {
  double *qbar;     // [b][Hkv][d][G]      (G: score rows per KV head)
  double *espill;   // [b][Hkv][S_pad][G]
  double *part;     // [b][Hkv][nchunk + 1][G][2]: (max, sum exp) per chunk, then
                    // of the normalisation tail
  uint64_t *keys;   // [b][Hkv][S_pad]
  uint32_t *hist;   // [b][Hkv][2048]
  float *opart;     // [b][Hkv][nchunk + 1][G][d]: attention output parts (optional output)
  uint64_t *cut;    // [b][Hkv][4]: the top-k cut (boundary prefix, its shift, keys of
                    // the boundary bucket still to take, whole-bucket flag and k)
  uint32_t *ecnt;   // [b][Hkv][nchunk]: keys above the cut (high 16 bits) and in the
                    // boundary bucket (low 16 bits) per chunk
  uint8_t *emark;   // [b][Hkv][nchunk][2][256]: per 8 consecutive keys, bit masks of
                    // the keys above the cut and of those in the boundary bucket
  int64_t S_pad;
  int nchunk;
};

constexpr int kScoreChunk = 2048;     // rows per scoring workgroup
constexpr int kHistBins = 2048;       // first-level radix bins (key >> 52)

size_t select_ws_bytes(int batch, int Hq, int Hkv, int d, int64_t max_seq_len,
                       SelectWs *layout, char *base);

// Largest number of score rows (query rows x query heads of a group) per KV
// head that the x-row selection takes.
constexpr int kMaxScoreRows = 512;

// Selection with x query rows of the block (the workspace laid out for
// V = x * G score rows per KV head in place of G). tail: [b][n_tail][Hkv][d]
// rows that enter every score row's (max, sum exp) but are never ranked
// (n_tail = 0: none).
hipError_t launch_select_xq(const herald_heads &hd, int batch, int block, int x,
                            const void *q_sel, const KvView &kv, const void *tail,
                            const void *tail_v, int n_tail, const int32_t *k_per_seq, int k_max,
                            int32_t *idx_out, void *o_out, const SelectWs &ws,
                            hipStream_t stream);

// Selection with the mean of the block's queries as the representative;
// tail as above.
// tail_v and o_out: the optional attention output of every score row over
// the cache and the tail, [b][V / G][Hq][d] (o_out null: none).
hipError_t launch_select(const herald_heads &hd, int batch, int block,
                         const void *q_sel, const KvView &kv, const void *tail,
                         const void *tail_v, int n_tail, const int32_t *k_per_seq, int k_max,
                         int32_t *idx_out, void *o_out, const SelectWs &ws,
                         hipStream_t stream);

}  // namespace herald
