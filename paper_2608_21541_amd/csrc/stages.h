// Argument blocks and host launchers of the kernel stages (internal).
#pragma once

#include <vector>

#include "common.h"

namespace certkv {

struct ScoreArgs {
  Geo g;
  certkv_tensor q, k;
  int32_t dtype;
  float* scores;
  double* ksum;
  float2* part;
  float* lse2;
  float* kpart;
  int32_t* flag;  // [U] units whose shift-free row sums left the safe range
  const float* lse_in;  // optional caller row log-sum-exp [L][B*w][Hq]
  float* lse_out;       // optional row log-sum-exp out, same layout
  int32_t keys_per_block;   // pass 1 (and its partials)
  int32_t nkb_max;
  int32_t keys_per_block2;  // pass 2 (and its key-sum partials)
  int32_t nkb2_max;
};
// Query tiles of 32 rows covering the M window rows, rounded up to a power of two.
inline int score_nqt(int M) {
  int t = 1;
  while (t * 32 < M) t *= 2;
  return t;
}
certkv_status run_score(const ScoreArgs& a, const SeqTab& st, int max_len, hipStream_t s);

struct SortArgs {
  Geo g;
  const float* scores;
  uint32_t *keysA, *keysB, *keys_out;
  int32_t *valsA, *valsB, *perm_out;
  double* ssum;
};
certkv_status run_sort(const SortArgs& a, const SeqTab& st, hipStream_t s);

struct CurveArgs {
  Geo g;
  const uint32_t* sorted_keys;
  const int32_t* perm;
  const double* ssum;
  certkv_tensor v;
  int32_t dtype;
  float* curves;
  double* vsum;
};
certkv_status run_curves(const CurveArgs& a, const SeqTab& st, hipStream_t s);

struct AllocArgs {
  Geo g;
  const float* curves;
  float* cmin;      // [U][nblk_max][2] minima of c over the two halves of each block
  float* cmaxb;     // [U][nblk_max] block maxima of c
  int32_t* cpos;    // [U][nblk_max] smallest position of the block minimum
  double* dmax;     // [U][nblk_max] block maxima of c(i+1) - c(i)
  int32_t nblk_max;
  int32_t steps;
  int32_t* budgets;
  int64_t* repairs;
  int32_t* sync;    // alloc_sync_words() words: cross-workgroup bisection (optional)
};
size_t alloc_sync_words();
certkv_status run_allocate(const AllocArgs& a, const SeqTab& st, hipStream_t s);

struct SelectArgs {
  Geo g;
  const float* scores;
  const uint32_t* sorted_keys;
  const int32_t* perm;
  int32_t* budgets;
  int64_t* kept_offsets;
  int64_t* packed_offsets;
  int32_t* kept_idx;
  int64_t capacity;
  double* evicted_sum;
  double* total_sum;
  uint64_t* bitmap;
  int32_t bm_stride;
};
certkv_status run_coverage(const Geo& g, const SeqTab& st, const float* scores,
                           const uint32_t* sorted_keys, double retain, int32_t* budgets,
                           hipStream_t s);
certkv_status run_clamp(const Geo& g, const SeqTab& st, int32_t* budgets, hipStream_t s);
certkv_status run_offsets(int64_t U, int32_t slot, const int32_t* budgets, int64_t* kept_offsets,
                          int64_t* packed_offsets, hipStream_t s);
certkv_status run_uniform_budgets(const Geo& g, const SeqTab& st, int32_t* budgets, hipStream_t s);
certkv_status run_select(const SelectArgs& a, const SeqTab& st, hipStream_t s);
certkv_status run_mask(const Geo& g, const std::vector<SeqTab>& tabs, const int64_t* kept_offsets,
                       const int32_t* kept_idx, uint8_t* mask, hipStream_t s);

struct TailArgs {
  Geo g;
  int32_t dtype;
  const float* scores;
  certkv_tensor k, v;
  const int64_t* kept_offsets;
  const int32_t* kept_idx;
  uint64_t* bitmap;
  int32_t bm_stride;
  int32_t nsplit;            // gather workgroups per unit
  double* kpart;             // [U][nsplit][2][D] partial kept sums
  double* mpart;             // [U][nsplit][3] partial masses (standalone path)
  const double* evicted_sum; // [U] from the selection pass, or NULL
  const double* total_sum;   // [U] from the selection pass, or NULL
  const double* ksum;
  const double* vsum;
  float* k_star;
  float* v_star;
  double* tail_mass;
  void* k_packed;
  void* v_packed;
  int32_t* pos_packed;
  bool do_tail, do_compact;
};
certkv_status run_bitmap(const TailArgs& a, const SeqTab& st, int64_t words_total, bool clear,
                         hipStream_t s);
certkv_status run_tail(const TailArgs& a, const SeqTab& st, hipStream_t s);
size_t score_smem_bytes(const Geo& g, int32_t dtype);

struct ClusterArgs {
  Geo g;
  int32_t dtype;
  int32_t m;                    // groups per head
  const int32_t* perm;          // [L][H][T] rank order of the pass
  const int32_t* budgets;       // [U]
  certkv_tensor k, v;
  void* kbar;                   // [U][m][d] in the cache dtype
  void* vbar;
  int32_t* count;               // [U][m]
  float* rk;                    // [U][m] key radii
  float* rv;                    // [U][m] value radii
  float* vmax_kept;             // [U]
};
certkv_status run_clusters(const ClusterArgs& a, const SeqTab& st, hipStream_t s);
certkv_status run_clusters_clear(float* vmax_kept, int64_t U, hipStream_t s);  // before run_clusters

// Optional clustered-tail terms of a decode (added in the combine).
struct DecodeClusters {
  int32_t m;                    // 0: none
  const uint16_t* kbar;         // [U][m][d] bf16
  const uint16_t* vbar;
  const int32_t* count;
  const float* rk;
  const float* rv;
  const float* vmax_kept;
  float* bound;                 // optional [L][B*tq][Hq] certificate (inf if it does not hold)
};

struct DecodeArgs {
  Geo g;
  int64_t U;
  int32_t tq;                   // new queries per sequence
  int32_t nsplit;               // 1024-key chunks of the longest segment allowed
  certkv_tensor q;              // [L][B*tq][Hq][d] bf16
  const void* k_packed;         // [P][d] bf16
  const void* v_packed;
  const int64_t* packed_offsets;
  float* part_o;                // [U][nsplit][mp][d]
  float2* part_ml;              // [U][nsplit][mp]
  int2* items;                  // [U * nsplit] work items (unit, chunk), built on device
  int32_t* item_count;          // their number
  float* out;                   // [L][B*tq][Hq][d]
  float* lse;                   // optional [L][B*tq][Hq]
  DecodeClusters cl;
};
// Query tiles of 32 rows for M decode rows, rounded up to a power of two.
inline int decode_nqt(int M) {
  int t = 1;
  while (t * 32 < M) t *= 2;
  return t;
}
certkv_status run_decode(const DecodeArgs& a, hipStream_t s);
size_t decode_partial_rows(int64_t U, int nsplit, int tq, int G);
int decode_nsplit(int max_len);

certkv_status run_packed_from_kept(int64_t U, int32_t slot, const int64_t* kept_offsets,
                                   int64_t* packed_offsets, hipStream_t s);
}  // namespace certkv
