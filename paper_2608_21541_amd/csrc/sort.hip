// Per-unit stable ordering of keys by score, descending, ties by position.
//
// One workgroup (16 waves) sorts one unit's segment with a least-significant-
// digit radix sort: 4 passes of 8-bit digits over the order-inverting key
// transform of the fp32 score (desc_key).  One counting pass first forms all
// four digit histograms with LDS atomics (and the fp64 sum of (s)_+, the
// normalizer of a_j).
// Each pass then walks the segment in tiles of 16 * 64 * R elements; wave w
// holds the R rounds of 64 consecutive elements at offset 64 R w:
//   rank     lanes with equal digits are found with 8 ballots; an element's
//            rank among equal digits of its wave is a per-wave LDS counter
//            plus mbcnt within the round (input order);
//   offsets  per digit, an exclusive scan over the waves, and per tile an
//            exclusive scan over the digits of the tile's digit counts (the
//            two run concurrently on different waves);
//   stage    every element is written to LDS at its digit-major position in
//            the tile (stable);
//   write    thread i stores staged element i to the digit's running bucket
//            offset plus its position inside the tile's run of that digit,
//            so consecutive threads write consecutive addresses.
// Ranking in input order and runs in tile order make every pass stable, so
// equal scores keep ascending position.  The next tile's elements are loaded
// while the current one is ranked.
#include <type_traits>

#include "stages.h"

namespace certkv {

constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kSortRounds = 8;
constexpr int kSortTile = kSortThreads * kSortRounds;  // 8192 elements

// Lanes of the wave whose 8-bit digit equals this lane's (among `valid`).
// Per bit, the lanes agreeing with this lane are the ballot of the bit when
// it is set here and its complement when it is clear: ballot ^ m with m the
// bit sign-extended from ~digit (0 or all ones), which keeps the selection a
// per-lane xor of a wave-uniform mask.
__device__ __forceinline__ uint64_t match_digit(uint32_t digit, bool valid) {
  const uint64_t v = __ballot(valid);
  uint32_t plo = (uint32_t)v, phi = (uint32_t)(v >> 32);
  const uint32_t nd = ~digit;
#pragma unroll
  for (int bit = 0; bit < 8; ++bit) {
    const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)nd, bit, 1);
    const uint64_t bb = __ballot(m == 0u);
    plo &= (uint32_t)bb ^ m;
    phi &= (uint32_t)(bb >> 32) ^ m;
  }
  return ((uint64_t)phi << 32) | plo;
}

__device__ __forceinline__ uint32_t count_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Exclusive scan of 256 counters by one wave (4 per lane), in place.
__device__ __forceinline__ void wave_scan256(uint32_t* v, int lane) {
  uint32_t c[4], run = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    c[j] = v[lane * 4 + j];
    run += c[j];
  }
  uint32_t incl = run;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  uint32_t excl = incl - run;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[lane * 4 + j] = excl;
    excl += c[j];
  }
}

__global__ __launch_bounds__(kSortThreads) void seg_sort_kernel(
    Geo g, SeqTab st, const float* __restrict__ scores, uint32_t* __restrict__ keysA,
    int32_t* __restrict__ valsA, uint32_t* __restrict__ keysB, int32_t* __restrict__ valsB,
    uint32_t* __restrict__ keys_out, int32_t* __restrict__ perm_out,
    double* __restrict__ ssum_out) {
  __shared__ uint32_t hist[4][256];
  __shared__ uint32_t bucket[256];      // running start of each digit's bucket
  __shared__ uint32_t tile_tot[2][256]; // digit counts of the tile, by tile parity
  __shared__ uint32_t tile_start[256];  // digit-major start inside the tile
  __shared__ uint32_t wave_cnt[kSortWaves][256];
  __shared__ uint32_t stage_key[kSortTile];
  __shared__ int32_t stage_val[kSortTile];
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
  // positions from wkeep on are the kept window: key 0 ranks them first
  const int wkeep = n - g.keep_w;

  for (int i = threadIdx.x; i < 4 * 256; i += kSortThreads) (&hist[0][0])[i] = 0u;
  for (int i = threadIdx.x; i < 2 * 256; i += kSortThreads) (&tile_tot[0][0])[i] = 0u;
  __syncthreads();

  // Counting pass: four digit histograms and the fp64 sum of (s)_+.  The
  // next tile's scores are loaded while the current one is counted.
  {
    double psum = 0.0;
    auto load_scores = [&](int t0, float (&x)[kSortRounds]) {
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
        const float v = scores[base + min(e, n - 1)];  // clamped: no branch around the load
        x[r] = e < n ? v : 0.f;
      }
    };
    float sv[kSortRounds], sn[kSortRounds];
    load_scores(0, sv);
    for (int t0 = 0; t0 < n; t0 += kSortTile) {
      load_scores(t0 + kSortTile, sn);  // unconditional: clamped reads, no branch
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
        const bool valid = e < n;
        if (valid && sv[r] > 0.f) psum += (double)sv[r];
        const uint32_t key = e >= wkeep ? 0u : desc_key(sv[r]);
        if (valid) {
#pragma unroll
          for (int p = 0; p < 3; ++p) atomicAdd(&hist[p][(key >> (8 * p)) & 255u], 1u);
        }
        // The top digit holds the score's sign and upper exponent bits, so a
        // wave sees few distinct values: one atomic per distinct digit
        // instead of one per lane on a handful of addresses.
        const uint32_t d3 = key >> 24;
        uint64_t todo = __ballot(valid);
        while (todo) {
          const int leader = __builtin_ctzll(todo);
          const uint32_t dl = __builtin_amdgcn_readlane(d3, leader);
          const uint64_t same = __ballot(d3 == dl) & todo;
          if (lane == leader) atomicAdd(&hist[3][dl], (uint32_t)__popcll(same));
          todo &= ~same;
        }
      }
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) sv[r] = sn[r];
    }
    psum = wave_sum(psum);
    if (lane == 0) dred[wave] = psum;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int w = 0; w < kSortWaves; ++w) tot += dred[w];
    ssum_out[u] = tot;
  }

  // One pass per digit, instantiated per pass so that its input (the scores
  // or the previous pass's output) is fixed at compile time and no branch
  // splits the tile loads.
  auto pass = [&](auto pass_tag) {
    constexpr int p = decltype(pass_tag)::value;
    const uint32_t* kin = p == 1 || p == 3 ? keysB : keysA;
    const int32_t* vin = p == 1 || p == 3 ? valsB : valsA;
    uint32_t* kout = (p == 0 || p == 2) ? keysB : (p == 1 ? keysA : keys_out);
    int32_t* vout = (p == 0 || p == 2) ? valsB : (p == 1 ? valsA : perm_out);
    const int sh = 8 * p;
    if (wave == 0) {
      for (int j = 0; j < 4; ++j) bucket[lane * 4 + j] = hist[p][lane * 4 + j];
      wave_scan256(bucket, lane);
    }
    // Loads through range-checked buffers: elements at or beyond n read as
    // zero, so no clamp or branch sits around them.  The first pass loads
    // the raw score bits and forms their radix keys (and the kept window's
    // zero keys) only when the tile is ranked, so that the next tile's loads
    // stay in flight meanwhile.
    const BufRsrc kin_r = make_rsrc(p == 0 ? (const void*)(scores + base) : (const void*)(kin + base),
                                    (uint32_t)n * 4u);
    const BufRsrc vin_r = make_rsrc(vin + base, (uint32_t)n * 4u);
    const BufRsrc kout_r = make_rsrc(kout + base, (uint32_t)n * 4u);
    const BufRsrc vout_r = make_rsrc(vout + base, (uint32_t)n * 4u);
    auto load = [&](int t0, uint32_t (&key)[kSortRounds], int32_t (&val)[kSortRounds]) {
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
        const uint32_t off = (uint32_t)e * 4u;
        if (p == 0) {
          key[r] = buf_load_u32(kin_r, off);
          val[r] = e;
        } else {
          key[r] = buf_load_u32(kin_r, off);
          val[r] = (int32_t)buf_load_u32(vin_r, off);
        }
      }
    };
    uint32_t key[kSortRounds], nkey[kSortRounds];
    int32_t val[kSortRounds], nval[kSortRounds];
    load(0, key, val);
    for (int t0 = 0; t0 < n; t0 += kSortTile) {
      const int tp = (t0 / kSortTile) & 1;  // tile parity
#pragma unroll
      for (int j = 0; j < 4; ++j) wave_cnt[wave][lane * 4 + j] = 0u;
      // prefetch, unconditionally (past the end the range check reads zeros),
      // so that no branch makes the compiler wait for it before the ranking
      load(t0 + kSortTile, nkey, nval);
      if (p == 0) {
#pragma unroll
        for (int r = 0; r < kSortRounds; ++r) {
          const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
          key[r] = e >= wkeep ? 0u : desc_key(__uint_as_float(key[r]));
        }
      }
      // rank within the wave
      uint32_t rank[kSortRounds];
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
        const bool ok = e < n;
        const uint32_t dg = (key[r] >> sh) & 255u;
        const uint64_t peers = match_digit(dg, ok);
        const uint32_t below = count_below(peers);
        uint32_t pre = 0;
        if (ok) pre = wave_cnt[wave][dg];
        rank[r] = pre + below;
        if (ok && below == 0) {
          const uint32_t c = (uint32_t)__popcll(peers);
          wave_cnt[wave][dg] = pre + c;
          atomicAdd(&tile_tot[tp][dg], c);
        }
      }
      __syncthreads();
      // per digit: exclusive scan over the waves (waves 1-4), over the digits
      // of the tile counts (wave 0) and the previous tile's advance of the
      // bucket offsets (waves 5-8; every wave is past that tile's writes),
      // concurrently.  The previous tile's counts are cleared for the tile
      // after this one.
      if (wave == 0) {
        for (int j = 0; j < 4; ++j) tile_start[lane * 4 + j] = tile_tot[tp][lane * 4 + j];
        wave_scan256(tile_start, lane);
      } else if (threadIdx.x >= 320 && threadIdx.x < 320 + 256) {
        const int d = threadIdx.x - 320;
        if (t0 > 0) bucket[d] += tile_tot[tp ^ 1][d];
        tile_tot[tp ^ 1][d] = 0u;
      } else if (threadIdx.x < 256 + 64) {
        const int d = threadIdx.x - 64;
        uint32_t c[kSortWaves];
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w) c[w] = wave_cnt[w][d];  // all reads in flight
        uint32_t run = 0;
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w) {
          wave_cnt[w][d] = run;
          run += c[w];
        }
      }
      __syncthreads();
      // stage in digit-major order
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        const int e = t0 + wave * 64 * kSortRounds + r * 64 + lane;
        if (e < n) {
          const uint32_t dg = (key[r] >> sh) & 255u;
          const uint32_t lp = tile_start[dg] + wave_cnt[wave][dg] + rank[r];
          stage_key[lp] = key[r];
          stage_val[lp] = val[r];
        }
      }
      __syncthreads();
      // coalesced write of the staged tile
      const int cnt = min(kSortTile, n - t0);
      {
        uint32_t kk[kSortRounds], dst[kSortRounds];
        int32_t vv[kSortRounds];
#pragma unroll
        for (int r = 0; r < kSortRounds; ++r) {
          const int i = threadIdx.x + r * kSortThreads;
          kk[r] = i < cnt ? stage_key[i] : 0u;
          vv[r] = i < cnt ? stage_val[i] : 0;
        }
#pragma unroll
        for (int r = 0; r < kSortRounds; ++r) {
          const int i = threadIdx.x + r * kSortThreads;
          const uint32_t d = (kk[r] >> sh) & 255u;
          dst[r] = bucket[d] + (uint32_t)i - tile_start[d];
        }
#pragma unroll
        for (int r = 0; r < kSortRounds; ++r) {
          const int i = threadIdx.x + r * kSortThreads;
          if (i < cnt) {
            buf_store_u32(kout_r, dst[r] * 4u, kk[r]);
            buf_store_u32(vout_r, dst[r] * 4u, (uint32_t)vv[r]);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < kSortRounds; ++r) {
        key[r] = nkey[r];
        val[r] = nval[r];
      }
    }
    // the last tile's counts (the other parity is already clear)
    if (threadIdx.x < 256) tile_tot[((n - 1) / kSortTile) & 1][threadIdx.x] = 0u;
    __syncthreads();  // the pass's output is the next pass's input
  };
  pass(std::integral_constant<int, 0>());
  pass(std::integral_constant<int, 1>());
  pass(std::integral_constant<int, 2>());
  pass(std::integral_constant<int, 3>());
  // Kept window: its keys sorted as 0 (ahead of every score) and so hold
  // ranks 0..w-1 in position order; give them their score keys back, which
  // the masses of the dispersion curves and the coverage prefix read.
  for (int t = threadIdx.x; t < g.keep_w; t += kSortThreads)
    keys_out[base + t] = desc_key(scores[base + n - g.keep_w + t]);
}

certkv_status run_sort(const SortArgs& a, const SeqTab& st, hipStream_t s) {
  CERTKV_LAUNCH("sort_segments", seg_sort_kernel, dim3(a.g.H * st.count, a.g.L), dim3(kSortThreads),
                0, s, a.g, st, a.scores, a.keysA, a.valsA, a.keysB, a.valsB, a.keys_out, a.perm_out,
                a.ssum);
  return CERTKV_OK;
}

}  // namespace certkv
