// Per-unit stable ordering of keys by score, descending, ties by position.
//
// One workgroup (16 waves) sorts one unit's segment with a least-significant-
// digit radix sort: 4 passes of 8-bit digits over the order-inverting key
// transform of the fp32 score (desc_key).  Stability is what makes equal
// scores keep ascending position, so every pass ranks elements in exactly
// their input order:
//   - a wave takes 256 consecutive elements of the tile in 4 rounds of 64;
//   - within a round, lanes with equal digits are found with 8 ballots and
//     ranked by mbcnt (lanes below them with the same digit);
//   - a per-wave, per-digit counter in LDS carries ranks across rounds;
//   - after the tile, an exclusive scan over waves per digit gives each wave's
//     offset, added to the digit's running bucket offset.
// All four digit histograms come from one counting pass that also sums
// (s)_+ in fp64 (the normalizer of the weights a_j).
#include "stages.h"

namespace certkv {

constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kSortRounds = 4;
constexpr int kSortTile = kSortThreads * kSortRounds;

// Lanes of the wave whose 8-bit digit equals this lane's (among `active`).
__device__ __forceinline__ uint64_t match_digit(uint32_t digit, bool valid) {
  uint64_t peers = __ballot(valid);
#pragma unroll
  for (int bit = 0; bit < 8; ++bit) {
    const bool set = (digit >> bit) & 1u;
    const uint64_t bb = __ballot(valid && set);
    peers &= set ? bb : ~bb;
  }
  return peers;
}

__device__ __forceinline__ uint32_t count_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__global__ __launch_bounds__(kSortThreads) void seg_sort_kernel(
    Geo g, SeqTab st, const float* __restrict__ scores, uint32_t* __restrict__ keysA,
    int32_t* __restrict__ valsA, uint32_t* __restrict__ keysB, int32_t* __restrict__ valsB,
    uint32_t* __restrict__ keys_out, int32_t* __restrict__ perm_out,
    double* __restrict__ ssum_out) {
  __shared__ uint32_t hist[4][256];
  __shared__ uint32_t bucket[256];
  __shared__ uint32_t tile_tot[256];
  __shared__ volatile uint32_t wave_cnt[kSortWaves][256];
  __shared__ double dred[kSortWaves];

  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t base = lht_base(g, l, h, st.start[bl]);
  const int64_t u = unit_index(g, l, b, h);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  for (int i = threadIdx.x; i < 4 * 256; i += kSortThreads) (&hist[0][0])[i] = 0u;
  __syncthreads();

  // Counting pass: four digit histograms and the fp64 sum of (s)_+.
  double psum = 0.0;
  for (int t0 = 0; t0 < n; t0 += kSortTile) {
#pragma unroll
    for (int r = 0; r < kSortRounds; ++r) {
      const int e = t0 + wave * 256 + r * 64 + lane;
      const bool valid = e < n;
      float s = valid ? scores[base + e] : 0.f;
      if (valid && s > 0.f) psum += (double)s;
      const uint32_t key = desc_key(s);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t dg = (key >> (8 * p)) & 255u;
        const uint64_t peers = match_digit(dg, valid);
        if (valid && count_below(peers) == 0) atomicAdd(&hist[p][dg], (uint32_t)__popcll(peers));
      }
    }
  }
  psum = wave_sum(psum);
  if (lane == 0) dred[wave] = psum;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int w = 0; w < kSortWaves; ++w) tot += dred[w];
    ssum_out[u] = tot;
  }

  const uint32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  for (int p = 0; p < 4; ++p) {
    uint32_t* kout = (p == 0 || p == 2) ? keysB : (p == 1 ? keysA : keys_out);
    int32_t* vout = (p == 0 || p == 2) ? valsB : (p == 1 ? valsA : perm_out);
    // Exclusive scan of the digit histogram -> bucket starts.
    __syncthreads();
    if (wave == 0) {
      uint32_t c[4], run = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = hist[p][lane * 4 + j];
        run += c[j];
      }
      uint32_t incl = run;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        uint32_t y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
      }
      uint32_t excl = incl - run;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bucket[lane * 4 + j] = excl;
        excl += c[j];
      }
    }
    __syncthreads();
    const int sh = 8 * p;
    for (int t0 = 0; t0 < n; t0 += kSortTile) {
#pragma unroll
      for (int j = 0; j < 4; ++j) wave_cnt[wave][lane * 4 + j] = 0u;
      uint32_t key[kSortRounds], dg[kSortRounds], rank[kSortRounds];
      int32_t val[kSortRounds];
      bool ok[kSortRounds];
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 256 + r * 64 + lane;
        ok[r] = e < n;
        if (p == 0) {
          key[r] = desc_key(ok[r] ? scores[base + e] : 0.f);
          val[r] = e;
        } else {
          key[r] = ok[r] ? kin[base + e] : 0u;
          val[r] = ok[r] ? vin[base + e] : 0;
        }
        dg[r] = (key[r] >> sh) & 255u;
        const uint64_t peers = match_digit(dg[r], ok[r]);
        const uint32_t below = count_below(peers);
        uint32_t pre = 0;
        if (ok[r]) pre = wave_cnt[wave][dg[r]];
        rank[r] = pre + below;
        if (ok[r] && below == 0) wave_cnt[wave][dg[r]] = pre + (uint32_t)__popcll(peers);
      }
      __syncthreads();
      if (threadIdx.x < 256) {
        uint32_t run = 0;
        for (int w = 0; w < kSortWaves; ++w) {
          uint32_t c = wave_cnt[w][threadIdx.x];
          wave_cnt[w][threadIdx.x] = run;
          run += c;
        }
        tile_tot[threadIdx.x] = run;
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const uint32_t dst = bucket[dg[r]] + wave_cnt[wave][dg[r]] + rank[r];
        if (ok[r] && dst < (uint32_t)n) {  // always true when the counts are right
          kout[base + dst] = key[r];
          vout[base + dst] = val[r];
        }
      }
      __syncthreads();
      if (threadIdx.x < 256) bucket[threadIdx.x] += tile_tot[threadIdx.x];
      __syncthreads();
    }
    kin = kout;
    vin = vout;
  }
}


certkv_status run_sort(const SortArgs& a, const SeqTab& st, hipStream_t s) {
  CERTKV_LAUNCH("sort_segments", seg_sort_kernel, dim3(a.g.H * st.count, a.g.L), dim3(kSortThreads),
                0, s, a.g, st, a.scores, a.keysA, a.valsA, a.keysB, a.valsB, a.keys_out, a.perm_out,
                a.ssum);
  return CERTKV_OK;
}

}  // namespace certkv
