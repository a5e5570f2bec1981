// Budget allocation (multiplier bisection + one-token repair) on gfx950.
//
// One workgroup per (layer, sequence).
//
// Bisection.  Each step needs, per head, the smallest b in [b_min, n-1]
// minimizing f(b) = fma(lambda, b, c(b)) in fp64 on the fp32 curve.  The scan
// is pruned exactly: for a run of ranks starting at b0 (clamped to b_min)
// with minimum cmin, every candidate has lambda*b + c(b) >= lambda*b0 + cmin,
// and round-to-nearest is monotone, so LB = fma(lambda, b0, cmin) <= f(b) on
// the run (the runs are the two 128-rank halves of each 256-rank block).  The block with the smallest bound is evaluated
// first (32 threads per head); every block whose (LB, b0) undercuts the best
// (f*, b*) lexicographically is then put on a candidate list and evaluated
// by the whole workgroup, one coalesced 256-wide row per block.  Blocks left
// out cannot hold the answer (ties favour smaller b), so the result equals the
// full scan.
//
// Repair.  Starting from b_h = b_h(lambda_hi), the method adds one token at a
// time to the head with the smallest marginal d_h(i) = c_h(i+1) - c_h(i)
// (ties: lowest head).  That greedy consumes the candidate increments in
// increasing order of the key (P_h(i), h, i), where P_h(i) is the running
// maximum of d_h over [b_h, i]: all increments keyed below a level are taken
// before any keyed at or above it, and within a level the lowest head runs
// first.  So the final budgets follow from the R-th smallest key, R = B_real -
// sum b_h: a bisection over the ordered bit patterns of fp64 keys finds it,
// counting per head with block-level running maxima (LDS) and one scan of the
// block where the running maximum crosses the threshold.
#include <type_traits>

#include "stages.h"

namespace certkv {

constexpr int kAllocThreads = 1024;
constexpr int kAllocWaves = kAllocThreads / 64;
constexpr int kHeadGroup = kAllocThreads / 32;  // heads handled concurrently (32 threads each)
constexpr int kCandCap = 1024;    // candidate blocks evaluated per round
constexpr int kBlk = 256;          // ranks per pruning block
constexpr int kLdsItems = 8192;    // H * blocks handled from LDS
constexpr int kRepairWin = 64;     // cached curve values per head (fallback repair)
constexpr int kRcStride = kBlk + 4;  // a cached curve block of the repair search: kBlk + 1 values
// Bisection across several workgroups per (layer, sequence): up to kTreeLev
// levels per pass, one workgroup per node of the level tree.
constexpr int kTreeLev = 3;
constexpr int kTreeMax = (1 << kTreeLev) - 1;
constexpr int kSyncGroups = 256;   // (layer, sequence) groups of one such launch at most
// sync words: ticket, pad, one word per group (unused), then per group and
// pass parity the nodes' budget sums tagged with their pass ((pass + 1) << 48
// | sum, int64) and argmin vectors (64 heads)
constexpr size_t kSyncCnt = 2 + kSyncGroups;
constexpr size_t kSyncSum = kSyncCnt;
constexpr size_t kSyncArg = kSyncSum + (size_t)kSyncGroups * 2 * kTreeMax * 2;
constexpr size_t kSyncWords = kSyncArg + (size_t)kSyncGroups * 2 * kTreeMax * 64;

size_t alloc_sync_words() { return kSyncWords; }

// Lanes below this one among those set in `mask`.
__device__ __forceinline__ uint32_t count_below64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// A curve value as the block statistics and the repair read it: unchanged
// when finite; NaN and +inf read as the largest finite float, -inf as its
// negative.  The bisection's candidate scans read the curves as they are (a
// NaN never wins a comparison), and a head left without an argmin starts the
// repair from b_min.  So with non-finite curves (a caller's, or from
// non-finite inputs) the budgets still lie in [b_min, n-1] and sum to B_real,
// meaningless as they are, and the status word reports the values.
__device__ __forceinline__ float cval(float x) {
  constexpr float kMax = 3.40282347e38f;  // the largest finite float
  return fmaxf(fminf(x, kMax), -kMax);
}

__device__ __forceinline__ bool lex_less(double f1, int b1, double f2, int b2) {
  return f1 < f2 || (f1 == f2 && b1 < b2);
}

struct BestFB {
  double f;
  int b;
};

// Minimum over each half-wave (lanes 0-31 and 32-63), in every lane of the
// half: DPP exchanges within rows of 16 lanes (lane ^ 1, lane ^ 2, then the
// mirrored lane within 8 and within 16: after the first steps the values are
// equal within the smaller groups, so a mirror pairs the groups as an xor
// would), then v_permlane16_swap pairs the two rows of each half.  Every lane
// of a half must be active.
__device__ __forceinline__ int half_min_i32(int x) {
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));
  x = min(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));
  const auto r = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)x, false, false);
  return min((int)r[0], (int)r[1]);
}

// The same minimum for floats (no NaN among the values).
__device__ __forceinline__ float half_min_f32(float x) {
  x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), 0xB1, 0xF, 0xF, false)));
  x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), 0x4E, 0xF, 0xF, false)));
  x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), 0x141, 0xF, 0xF, false)));
  x = fminf(x, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), 0x140, 0xF, 0xF, false)));
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fminf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Lexicographic (f, b) minimum reductions, carrying a float c of the winning
// lane (the order is total on (f, b), so the result does not depend on the
// pairing).  The exchanges are those of half_min_i32, plus v_permlane32_swap
// for the whole wave; every lane of the reduced group must be active.
__device__ __forceinline__ void lex_take(double& f, int& b, float& c, double fo, int bo, float co) {
  if (lex_less(fo, bo, f, b)) {
    f = fo;
    b = bo;
    c = co;
  }
}

template <int CTL>
__device__ __forceinline__ void lex_dpp(double& f, int& b, float& c) {
  const uint64_t u = (uint64_t)__double_as_longlong(f);
  const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)u, (int)(uint32_t)u, CTL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(u >> 32), (int)(uint32_t)(u >> 32), CTL,
                                             0xF, 0xF, false);
  const int bo = __builtin_amdgcn_update_dpp(b, b, CTL, 0xF, 0xF, false);
  const int co = __builtin_amdgcn_update_dpp(__float_as_int(c), __float_as_int(c), CTL, 0xF, 0xF, false);
  const double fo = __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
  lex_take(f, b, c, fo, bo, __int_as_float(co));
}

// One exchange between the pairs of 16-lane rows of each half (W = 16) or
// between the halves (W = 32): both candidates arrive in every lane.
template <int W>
__device__ __forceinline__ void lex_swap(double& f, int& b, float& c) {
  const uint64_t u = (uint64_t)__double_as_longlong(f);
  const uint32_t lo = (uint32_t)u, hi = (uint32_t)(u >> 32);
  const uint32_t bu = (uint32_t)b, cu = __float_as_uint(c);
  auto sw = [](uint32_t x) {
    if constexpr (W == 16)
      return __builtin_amdgcn_permlane16_swap(x, x, false, false);
    else
      return __builtin_amdgcn_permlane32_swap(x, x, false, false);
  };
  const auto rl = sw(lo), rh = sw(hi), rb = sw(bu), rc = sw(cu);
  f = __longlong_as_double((long long)(((uint64_t)rh[0] << 32) | rl[0]));
  b = (int)rb[0];
  c = __uint_as_float(rc[0]);
  lex_take(f, b, c, __longlong_as_double((long long)(((uint64_t)rh[1] << 32) | rl[1])), (int)rb[1],
           __uint_as_float(rc[1]));
}

// over `WIDTH` lanes: 32 (each half-wave) or 64 (the wave)
template <int WIDTH>
__device__ __forceinline__ void lexmin_fbc(double& f, int& b, float& c) {
  lex_dpp<0xB1>(f, b, c);   // lane ^ 1
  lex_dpp<0x4E>(f, b, c);   // lane ^ 2
  lex_dpp<0x141>(f, b, c);  // mirrored within 8
  lex_dpp<0x140>(f, b, c);  // mirrored within 16
  lex_swap<16>(f, b, c);
  if constexpr (WIDTH == 64) lex_swap<32>(f, b, c);
}

__device__ __forceinline__ BestFB half_wave_min(double f, int b) {
  float c = 0.f;
  lexmin_fbc<32>(f, b, c);
  return BestFB{f, b};
}

__device__ __forceinline__ BestFB wave_lexmin(double f, int b) {
  float c = 0.f;
  lexmin_fbc<64>(f, b, c);
  return BestFB{f, b};
}

// Monotone map between fp64 values and unsigned keys (total order of doubles).
__device__ __forceinline__ uint64_t dkey(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u & 0x8000000000000000ull) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double dval(uint64_t k) {
  const uint64_t u = (k & 0x8000000000000000ull) ? (k & 0x7fffffffffffffffull) : ~k;
  return __longlong_as_double((long long)u);
}

// Per-block statistics of the curves: minimum of c over each 128-rank half of
// each 256-rank block (+inf where a half is past the end), maximum of c over
// the block, the smallest position holding the block minimum, and the
// maximum marginal d(i) = c(i+1) - c(i) (fp64) over the i of the block with
// i <= n-2.  One wave per kBsBlocks consecutive blocks, the loads of all of
// them in flight at once (positions clamped into the segment, masked where
// used); lane L covers positions 4L..4L+3 of a block (lanes 0-31 the first
// half), and the wave reductions are DPP and lane-row exchanges.
constexpr int kBsBlocks = 8;

template <typename T, typename F>
__device__ __forceinline__ T wave_reduce_dpp(T x, F op) {
  static_assert(sizeof(T) == 4, "32-bit values");
  auto dpp = [&](auto ctl) {
    return __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, x), __builtin_bit_cast(int, x),
                                                             decltype(ctl)::value, 0xF, 0xF, false));
  };
  x = op(x, dpp(std::integral_constant<int, 0xB1>()));
  x = op(x, dpp(std::integral_constant<int, 0x4E>()));
  x = op(x, dpp(std::integral_constant<int, 0x141>()));
  x = op(x, dpp(std::integral_constant<int, 0x140>()));
  // (the swap results are read into scalars before the bit casts: a bit cast
  // applied to a subscripted element of the result vector compiled to the
  // first element for both subscripts)
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const uint32_t a0 = r16[0], a1 = r16[1];
  x = op(__builtin_bit_cast(T, a0), __builtin_bit_cast(T, a1));
  const uint32_t v = __builtin_bit_cast(uint32_t, x);
  const auto r32 = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  const uint32_t b0 = r32[0], b1 = r32[1];
  return op(__builtin_bit_cast(T, b0), __builtin_bit_cast(T, b1));
}

__global__ __launch_bounds__(256) void curve_blockstats_kernel(Geo g, SeqTab st, int32_t nblk_max,
                                                               const float* __restrict__ curves,
                                                               float* __restrict__ cmin,
                                                               float* __restrict__ cmaxb,
                                                               int32_t* __restrict__ cpos,
                                                               double* __restrict__ dmax,
                                                               int32_t* __restrict__ sync, int32_t nsync) {
  // the allocation's exchange words (ticket, tagged sums) start at zero: the
  // first workgroup clears them for the allocation kernel launched next
  if (sync && blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < nsync; i += 256) sync[i] = 0;
  const int per_unit = (nblk_max + 4 * kBsBlocks - 1) / (4 * kBsBlocks);
  const int wb = blockIdx.x % per_unit;
  const int hb = blockIdx.x / per_unit;
  const int h = hb % g.H;
  const int bl = hb / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int n = st.len[bl];
  const int nblk = (n + kBlk - 1) / kBlk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int k0 = (wb * 4 + wave) * kBsBlocks;
  if (k0 >= nblk) return;
  const int64_t u = unit_index(g, l, st.first + bl, h);
  const float* ch = curves + lht_base(g, l, h, st.start[bl]);
  float c[kBsBlocks][5];
#pragma unroll
  for (int j = 0; j < kBsBlocks; ++j) {
    const int i0 = (k0 + j) * kBlk + lane * 4;
#pragma unroll
    for (int e = 0; e < 5; ++e) c[j][e] = ch[min(i0 + e, n - 1)];
  }
  // a caller's non-finite curve values: reported, then read as cval() reads them
  bool bad = false;
#pragma unroll
  for (int j = 0; j < kBsBlocks; ++j) {
#pragma unroll
    for (int e = 0; e < 5; ++e) {
      bad |= !isfinite(c[j][e]);
      c[j][e] = cval(c[j][e]);
    }
  }
  if (__ballot(bad) != 0ull && lane == 0) report_nonfinite(g);
#pragma unroll
  for (int j = 0; j < kBsBlocks; ++j) {
    const int k = k0 + j;
    if (k >= nblk) break;
    const int i0 = k * kBlk + lane * 4;
    float mn = INFINITY, mx = -INFINITY;
    int pmn = 0x7fffffff;
    double dm = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (i0 + e < n) {
        if (c[j][e] < mn) {
          mn = c[j][e];
          pmn = i0 + e;
        }
        mx = fmaxf(mx, c[j][e]);
      }
      if (i0 + e <= n - 2) dm = fmax(dm, (double)c[j][e + 1] - (double)c[j][e]);
    }
    const float mhalf = half_min_f32(mn);
    // (min c, smallest position): the lexicographic minimum of (c, position)
    // (min c, smallest position): the smallest position holding the minimum
    const float mnw = wave_reduce_dpp(mn, [](float a, float b) { return fminf(a, b); });
    const int pw = wave_reduce_dpp(mn == mnw ? pmn : 0x7fffffff, [](int a, int b) { return min(a, b); });
    mx = wave_reduce_dpp(mx, [](float a, float b) { return fmaxf(a, b); });
    dm = wave_max(dm);
    if ((lane & 31) == 0) cmin[(u * nblk_max + k) * 2 + (lane >> 5)] = mhalf;
    if (lane == 0) {
      cmaxb[u * nblk_max + k] = mx;
      cpos[u * nblk_max + k] = pw;
      dmax[u * nblk_max + k] = dm;
    }
  }
}

__global__ __launch_bounds__(kAllocThreads) void allocate_kernel(
    Geo g, SeqTab st, const float* __restrict__ curves, const float* __restrict__ cmin,
    const float* __restrict__ cmaxb, const int32_t* __restrict__ cpos,
    const double* __restrict__ dmax, int32_t nblk_max, int32_t steps,
    int32_t* __restrict__ budgets, int64_t* __restrict__ stats, int32_t K, int32_t* sync) {
  // 64 KB of LDS: the half-block minima during the bisection, the
  // block-level running maxima of the marginals during the repair.
  __shared__ __align__(16) unsigned char pool[kLdsItems * 8];
  float2* mcache = reinterpret_cast<float2*>(pool);  // half-block minima
  double* pbm = reinterpret_cast<double*>(pool);
  __shared__ int32_t cand[kCandCap];
  __shared__ double fbest[64];
  __shared__ int32_t bbest[64], kstar[64];
  __shared__ float cbest[64], cprev[64];  // curve values at bbest and bprev
  __shared__ int32_t bprev[64];           // previous argmin (-1: none)
  // One region for three phases: the smallest position of each block's
  // minimum (bisection), the repair search's cached curve blocks, one per
  // (threshold, head) half-wave, and the sequential repair's curve windows.
  constexpr size_t kAuxA = (size_t)kLdsItems * 4, kAuxB = (size_t)kHeadGroup * kRcStride * 4,
                   kAuxC = (size_t)64 * (kRepairWin + 1) * 4;
  constexpr size_t kAux = kAuxA > kAuxB ? (kAuxA > kAuxC ? kAuxA : kAuxC) : (kAuxB > kAuxC ? kAuxB : kAuxC);
  __shared__ __align__(16) unsigned char aux[kAux];
  int32_t* mpos = reinterpret_cast<int32_t*>(aux);
  float* rcache = reinterpret_cast<float*>(aux);
  float(*win)[kRepairWin + 1] = reinterpret_cast<float(*)[kRepairWin + 1]>(aux);
  __shared__ int32_t rkey[kHeadGroup];
  __shared__ int32_t sfirst;  // (head << 16) | block of each cached block (-1: none)
  __shared__ float cres_c[kCandCap];
  __shared__ int32_t bcur[64], bhi[64];
  __shared__ double redf[kAllocWaves];
  __shared__ double cres_f[kCandCap];
  __shared__ int32_t cres_b[kCandCap];
  __shared__ int32_t ncand, scan_pos;
  __shared__ int64_t cnt_lt[64], cnt_le[64];
  __shared__ int64_t cnt_j[64];  // per (threshold, head) counts of the repair search
  __shared__ double tlam[kTreeMax], tlo[kTreeMax], thi[kTreeMax];  // node multipliers
  __shared__ int64_t tsum[kTreeMax];                                // node budget sums
  __shared__ int32_t ticket;

  // With K > 1 workgroups per (layer, sequence), groups are formed from an
  // atomic ticket in arrival order: a workgroup waits only for the others of
  // its group, and the lowest unfinished group either has every member
  // started or holds every started workgroup, so groups always complete.
  int bl, l, node = 0, grp = 0;
  if (K > 1) {
    if (threadIdx.x == 0) ticket = atomicAdd(&sync[0], 1);
    __syncthreads();
    grp = ticket / K;
    node = ticket - grp * K;
    bl = grp % st.count;
    l = grp / st.count;
  } else {
    bl = blockIdx.x;
    l = blockIdx.y;
  }
  if (bl >= st.count || l >= g.L) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int64_t B_real = st.b_real[bl];
  const int bmin = st.b_min[bl];
  const int H = g.H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int sub = tid & 31;
  const int hg = tid >> 5;
  const int nblk = (n + kBlk - 1) / kBlk;
  const int kfirst = bmin / kBlk;
  const bool fast = H * nblk <= kLdsItems;
  const uint64_t t_start = wall_clock64();

  // lambda_hi = 2 max c + 1 over every head and b in [0, n-1]
  double cm = 0.0;
  for (int i = tid; i < H * nblk; i += kAllocThreads) {
    const int h = i / nblk, k = i % nblk;
    cm = fmax(cm, (double)cmaxb[unit_index(g, l, b, h) * nblk_max + k]);
  }
  cm = wave_max(cm);
  if (lane == 0) redf[wave] = cm;
  if (fast) {
    for (int i = tid; i < H * nblk; i += kAllocThreads) {
      const int h = i / nblk, k = i % nblk;
      mcache[i] = reinterpret_cast<const float2*>(cmin)[unit_index(g, l, b, h) * nblk_max + k];
      mpos[i] = cpos[unit_index(g, l, b, h) * nblk_max + k];
    }
  }
  if (tid < 64) bprev[tid] = -1;
  __syncthreads();
  for (int w = 0; w < kAllocWaves; ++w) cm = fmax(cm, redf[w]);
  double lo = 0.0, hi = 2.0 * cm + 1.0;

  // minimum of c over block k of head h
  auto mh_at = [&](int h, int k) -> float {
    const float2 m = fast ? mcache[h * nblk + k]
                          : reinterpret_cast<const float2*>(cmin)[unit_index(g, l, b, h) * nblk_max + k];
    return fminf(m.x, m.y);
  };
  // Whether block k of head h (LDS item i) may hold a point undercutting the
  // head's best (f*, b*): per half, every point b of it has (f(b), b) >=
  // (fma(lam, b0, min c), b0) lexicographically.
  auto undercuts = [&](int i, int h, int k, double lam) -> bool {
    const float2 m = mcache[i];
    const int b0a = max(k * kBlk, bmin), b0b = max(k * kBlk + kBlk / 2, bmin);
    const bool a = k * kBlk + kBlk / 2 - 1 >= bmin &&
                   lex_less(fma(lam, (double)b0a, (double)m.x), b0a, fbest[h], bbest[h]);
    return a || lex_less(fma(lam, (double)b0b, (double)m.y), b0b, fbest[h], bbest[h]);
  };

  // Per head, the block with the smallest bound fma(lambda, b0, min c) is
  // evaluated exactly by 32 threads: (fbest, bbest) is then an exact upper
  // bound of the head's minimum and kstar its block.
  auto best_bound = [&](double lam) {
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        const float* ch = curves + lht_base(g, l, h, tok0);
        double lbest = INFINITY;
        int kb_ = 0x7fffffff;
        for (int k = kfirst + sub; k < nblk; k += 32) {
          const int b0 = max(k * kBlk, bmin);
          const double lb = fma(lam, (double)b0, (double)mh_at(h, k));
          if (lex_less(lb, k, lbest, kb_)) {
            lbest = lb;
            kb_ = k;
          }
        }
        const int ks = half_wave_min(lbest, kb_).b;
        double f = INFINITY;
        int bb = 0x7fffffff;
        const int lo_b = max(ks * kBlk, bmin), hi_b = min(ks * kBlk + kBlk - 1, n - 1);
        float cv[kBlk / 32];
#pragma unroll
        for (int i = 0; i < kBlk / 32; ++i) {
          const int x = ks * kBlk + sub + 32 * i;
          cv[i] = (x >= lo_b && x <= hi_b) ? ch[x] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < kBlk / 32; ++i) {
          const int x = ks * kBlk + sub + 32 * i;
          if (x >= lo_b && x <= hi_b) {
            const double v = fma(lam, (double)x, (double)cv[i]);
            if (lex_less(v, x, f, bb)) {
              f = v;
              bb = x;
            }
          }
        }
        const BestFB r = half_wave_min(f, bb);
        if (sub == 0) {
          fbest[h] = r.f;
          bbest[h] = r.b;
          kstar[h] = ks;
        }
      }
    }
    __syncthreads();
  };

  // argmin over [bmin, n-1] of fma(lam, b, c_h(b)) for every head -> out[h],
  // for problems whose block minima do not fit in LDS: per-head pruned scans
  auto evaluate_scan = [&](double lam, int32_t* out) {
    best_bound(lam);
    {
      // every other block re-checked by its head's 32 threads
      for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
        const int h = h0 + hg;
        if (h < H) {
          const float* ch = curves + lht_base(g, l, h, tok0);
          double f = fbest[h];
          int bb = bbest[h];
          for (int k = kfirst + sub; k < nblk; k += 32) {
            if (k == kstar[h]) continue;
            const int b0 = max(k * kBlk, bmin);
            const double lb = fma(lam, (double)b0, (double)mh_at(h, k));
            if (!lex_less(lb, b0, f, bb)) continue;
            const int hi_b = min(k * kBlk + kBlk - 1, n - 1);
            for (int x = b0; x <= hi_b; ++x) {
              const double v = fma(lam, (double)x, (double)ch[x]);
              if (lex_less(v, x, f, bb)) {
                f = v;
                bb = x;
              }
            }
          }
          const BestFB r = half_wave_min(f, bb);
          if (sub == 0) {
            fbest[h] = r.f;
            bbest[h] = r.b;
          }
        }
      }
      __syncthreads();
    }
    if (tid < H) out[tid] = bbest[tid];
    __syncthreads();
  };

  // The same argmin with the block minima in LDS, in rounds of at most
  // kCandCap candidate blocks (used when one round cannot hold them all).
  //  1. per head, the block with the smallest bound is evaluated exactly
  //     (32 threads per head): an exact upper bound (f*, b*) of the minimum;
  //  2. every other block whose bound undercuts (f*, b*) is a candidate;
  //     candidates of all heads are gathered (up to kCandCap per round) and
  //     evaluated one block per wave, all loads of a round in flight at once;
  //  3. per head, the smallest (f, b) over its candidates and (f*, b*).
  // Blocks left out cannot hold the answer (ties favour smaller b), so the
  // result is the full scan's.
  auto evaluate_rounds = [&](double lam, int32_t* out) {
    best_bound(lam);
    if (tid == 0) scan_pos = 0;
    __syncthreads();
    const int nitems = H * nblk;
    while (true) {
      // gather candidates from scan_pos on, until the list is full
      if (tid == 0) ncand = 0;
      __syncthreads();
      const int start = scan_pos;
      int stop = nitems;
      for (int i0 = start; i0 < nitems; i0 += kAllocThreads) {
        const int i = i0 + tid;
        bool take = false;
        int h = 0, k = 0;
        if (i < nitems) {
          h = i / nblk;
          k = i - h * nblk;
          if (k >= kfirst && k != kstar[h]) take = undercuts(i, h, k, lam);
        }
        const uint64_t m = __ballot(take);
        int slot0 = 0;
        if (lane == 0 && m) slot0 = atomicAdd(&ncand, __popcll(m));
        slot0 = __builtin_amdgcn_readfirstlane(slot0);
        const int slot = slot0 + (int)count_below64(m);
        if (take && slot < kCandCap) cand[slot] = (h << 16) | k;
        __syncthreads();
        if (ncand > kCandCap) {  // overflow: this sweep is scanned again next round
          stop = i0;
          break;
        }
        if (ncand == kCandCap) {  // full: resume after this sweep
          stop = i0 + kAllocThreads;
          break;
        }
      }
      __syncthreads();
      const int C = min(ncand, kCandCap);
      // evaluate: one candidate block per wave, up to 4 per wave per batch
      for (int c0 = wave; c0 < C; c0 += 4 * kAllocWaves) {
        float cv[4][kBlk / 64];
        int it[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = c0 + q * kAllocWaves;
          it[q] = c < C ? cand[c] : -1;
          const int hq = it[q] < 0 ? 0 : (it[q] >> 16), kq = it[q] < 0 ? 0 : (it[q] & 0xffff);
          const float* ch = curves + lht_base(g, l, hq, tok0);
#pragma unroll
          for (int e = 0; e < kBlk / 64; ++e) {
            const int x = kq * kBlk + lane + 64 * e;
            cv[q][e] = (it[q] >= 0 && x >= bmin && x <= n - 1) ? ch[x] : 0.f;
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (it[q] < 0) continue;
          const int kq = it[q] & 0xffff;
          double f = INFINITY;
          int bb = 0x7fffffff;
#pragma unroll
          for (int e = 0; e < kBlk / 64; ++e) {
            const int x = kq * kBlk + lane + 64 * e;
            if (x >= bmin && x <= n - 1) {
              const double v = fma(lam, (double)x, (double)cv[q][e]);
              if (lex_less(v, x, f, bb)) {
                f = v;
                bb = x;
              }
            }
          }
          const BestFB r = wave_lexmin(f, bb);
          if (lane == 0) {
            cres_f[c0 + q * kAllocWaves] = r.f;
            cres_b[c0 + q * kAllocWaves] = r.b;
          }
        }
      }
      __syncthreads();
      // per head: fold the candidates' minima into (f*, b*), 32 threads a head
      for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
        const int h = h0 + hg;
        if (h < H) {
          double f = INFINITY;
          int bb = 0x7fffffff;
          for (int c = sub; c < C; c += 32) {
            if ((cand[c] >> 16) == h && lex_less(cres_f[c], cres_b[c], f, bb)) {
              f = cres_f[c];
              bb = cres_b[c];
            }
          }
          const BestFB r = half_wave_min(f, bb);
          if (sub == 0 && lex_less(r.f, r.b, fbest[h], bbest[h])) {
            fbest[h] = r.f;
            bbest[h] = r.b;
          }
        }
      }
      if (tid == 0) scan_pos = stop;
      __syncthreads();
      if (stop >= nitems) break;
    }
    if (tid < H) {
      out[tid] = bbest[tid];
      bprev[tid] = -1;
    }
    __syncthreads();
  };

  // The argmin with an upper bound that needs no global load: per head the
  // best of (a) the first position of each block's minimum, for blocks whose
  // minimum lies at or after b_min (an actual point of the curve, its value
  // in LDS), and (b) the previous argmin with its curve value.  Every block
  // whose bound undercuts it is a candidate, gathered in one sweep and
  // evaluated one block per wave; if more than kCandCap qualify, the rounds
  // above take over.  As there, blocks left out cannot hold the answer.
  auto evaluate_fast = [&](double lam, int32_t* out) {
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        double f = INFINITY;
        int bb = 0x7fffffff;
        float cb = 0.f;
#pragma unroll 4
        for (int k = kfirst + sub; k < nblk; k += 32) {
          const int p = mpos[h * nblk + k];
          if (p >= bmin) {
            const float cv = fminf(mcache[h * nblk + k].x, mcache[h * nblk + k].y);
            const double v = fma(lam, (double)p, (double)cv);
            if (lex_less(v, p, f, bb)) {
              f = v;
              bb = p;
              cb = cv;
            }
          }
        }
        if (sub == 0 && bprev[h] >= 0) {
          const double v = fma(lam, (double)bprev[h], (double)cprev[h]);
          if (lex_less(v, bprev[h], f, bb)) {
            f = v;
            bb = bprev[h];
            cb = cprev[h];
          }
        }
        lexmin_fbc<32>(f, bb, cb);
        if (sub == 0) {
          fbest[h] = f;
          bbest[h] = bb;
          cbest[h] = cb;
        }
      }
    }
    if (tid == 0) ncand = 0;
    __syncthreads();
    const int nitems = H * nblk;
    for (int i0 = 0; i0 < nitems; i0 += kAllocThreads) {
      const int i = i0 + tid;
      bool take = false;
      int h = 0, k = 0;
      if (i < nitems) {
        h = i / nblk;
        k = i - h * nblk;
        if (k >= kfirst) take = undercuts(i, h, k, lam);
      }
      const uint64_t m = __ballot(take);
      int slot0 = 0;
      if (lane == 0 && m) slot0 = atomicAdd(&ncand, __popcll(m));
      slot0 = __builtin_amdgcn_readfirstlane(slot0);
      const int slot = slot0 + (int)count_below64(m);
      if (take && slot < kCandCap) cand[slot] = (h << 16) | k;
    }
    __syncthreads();
    const int C = ncand;
    if (C > kCandCap) {
      evaluate_rounds(lam, out);
      return;
    }
    // evaluate: each wave takes a run of `per` consecutive candidates (up to
    // 9, the most whose loads fit in flight in the registers), the
    // candidates spread evenly over the waves; the sweep lists them in (head, block) order, so a run
    // mostly belongs to one head: lanes keep a running best over the run's
    // positions and the wave reduces once per head change, recording the
    // result at that head's last candidate of the run (the others get +inf)
    constexpr int QB = 9;
    const int per = min(QB, (C + kAllocWaves - 1) / kAllocWaves);
    for (int c0 = wave * per; c0 < C; c0 += per * kAllocWaves) {
      float cv[QB][kBlk / 64];
      int it[QB];
#pragma unroll
      for (int q = 0; q < QB; ++q) {
        const int c = c0 + q;
        it[q] = (q < per && c < C) ? cand[c] : -1;
        const int hq = it[q] < 0 ? 0 : (it[q] >> 16), kq = it[q] < 0 ? 0 : (it[q] & 0xffff);
        const float* ch = curves + lht_base(g, l, hq, tok0);
#pragma unroll
        for (int e = 0; e < kBlk / 64; ++e) {
          const int x = kq * kBlk + lane + 64 * e;
          cv[q][e] = (it[q] >= 0 && x >= bmin && x <= n - 1) ? ch[x] : 0.f;
        }
      }
      double f = INFINITY;
      int bb = 0x7fffffff;
      float cb = 0.f;
#pragma unroll
      for (int q = 0; q < QB; ++q) {
        if (it[q] < 0) break;
        const int kq = it[q] & 0xffff;
#pragma unroll
        for (int e = 0; e < kBlk / 64; ++e) {
          const int x = kq * kBlk + lane + 64 * e;
          if (x >= bmin && x <= n - 1) {
            const double v = fma(lam, (double)x, (double)cv[q][e]);
            if (lex_less(v, x, f, bb)) {
              f = v;
              bb = x;
              cb = cv[q][e];
            }
          }
        }
        const bool last = q + 1 == QB || it[q + 1] < 0 || (it[q + 1] >> 16) != (it[q] >> 16);
        if (last) {
          lexmin_fbc<64>(f, bb, cb);
          if (lane == 0) {
            cres_f[c0 + q] = f;
            cres_b[c0 + q] = bb;
            cres_c[c0 + q] = cb;
          }
          f = INFINITY;
          bb = 0x7fffffff;
          cb = 0.f;
        } else if (lane == 0) {
          cres_f[c0 + q] = INFINITY;
          cres_b[c0 + q] = 0x7fffffff;
        }
      }
    }
    __syncthreads();
    // per head: fold the candidates' minima into (f*, b*), 32 threads a head
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        double f = fbest[h];
        int bb = bbest[h];
        float cb = cbest[h];
        for (int c = sub; c < C; c += 32) {
          if ((cand[c] >> 16) == h && lex_less(cres_f[c], cres_b[c], f, bb)) {
            f = cres_f[c];
            bb = cres_b[c];
            cb = cres_c[c];
          }
        }
        lexmin_fbc<32>(f, bb, cb);
        if (sub == 0) {
          out[h] = bb;
          bprev[h] = bb;
          cprev[h] = cb;
        }
      }
    }
    __syncthreads();
  };
  auto evaluate = [&](double lam, int32_t* out) {
    if (fast)
      evaluate_fast(lam, out);
    else
      evaluate_scan(lam, out);
  };

  // Bisection on lambda: lambda = (lo + hi) / 2, then lo = lambda if the
  // budgets at lambda sum above B_real, else hi = lambda (and bhi = the
  // budgets there).
  // The budgets at the initial lambda_hi are needed only when no step lowers
  // it; they are then evaluated after the steps.
  bool have_bhi = false;
  if (K <= 1) {
    for (int t = 0; t < steps; ++t) {
      const double lam = (lo + hi) / 2.0;
      evaluate(lam, bcur);
      int64_t sum = 0;
      for (int h = 0; h < H; ++h) sum += bcur[h];
      if (sum > B_real) {
        lo = lam;
      } else {
        hi = lam;
        have_bhi = true;
        if (tid < H) bhi[tid] = bcur[tid];
      }
      __syncthreads();
    }
    if (!have_bhi) evaluate(hi, bhi);
  } else {
    // The same steps, lev at a time: the multipliers of the next lev steps
    // form a binary tree (node i's children 2i+1 after hi = lambda_i and
    // 2i+2 after lo = lambda_i), each computed from its interval exactly as
    // the step-by-step bisection would.  The group's workgroup `node`
    // evaluates node `node`, the sums are exchanged through global memory,
    // and every workgroup then follows the same path down the tree.  Only
    // node 0 keeps bhi and goes on to the repair.
    const int lev_max = 31 - __clz(K + 1);
    int64_t* xsum = reinterpret_cast<int64_t*>(sync + kSyncSum) + (size_t)grp * 2 * kTreeMax;
    int32_t* xarg = sync + kSyncArg + (size_t)grp * 2 * kTreeMax * 64;
    int t = 0, pass = 0;
    // node 0: the argmins of the last node whose sum lowered lambda_hi, kept
    // in flight in registers while the next pass evaluates (the release of
    // the next publication waits for them) and stored once after the loop
    int32_t arg_hi = 0;
    while (t < steps) {
      const int lv = min(lev_max, steps - t);
      const int nl = (1 << lv) - 1;
      const int par = pass & 1;
      if (tid == 0) {
        tlo[0] = lo;
        thi[0] = hi;
        for (int i = 0; i < nl; ++i) {
          tlam[i] = (tlo[i] + thi[i]) / 2.0;
          if (2 * i + 2 < nl) {
            tlo[2 * i + 1] = tlo[i];
            thi[2 * i + 1] = tlam[i];
            tlo[2 * i + 2] = tlam[i];
            thi[2 * i + 2] = thi[i];
          }
        }
      }
      __syncthreads();
      if (node < nl) {
        evaluate(tlam[node], bcur);
        if (tid < H)
          __hip_atomic_store(&xarg[(par * kTreeMax + node) * 64 + tid], bcur[tid],
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      // Exchange.  Each evaluating node publishes its budget sum tagged with
      // the pass, released after its argmins (ordered before it by the
      // barrier); lanes 0..nl-1 of wave 0 poll one node's slot each with
      // coherent (agent-scope atomic) loads until every tag shows this pass,
      // and so hold the sums when the wait ends.  No acquire fence is needed
      // (the argmins are read with the same loads; an agent-scope acquire
      // would also invalidate the compute die's L2, which holds the curve
      // blocks the next evaluation rereads).  Slots alternate by pass parity:
      // a node publishes pass p + 2 only after it has seen every node's pass
      // p + 1, which each node publishes after reading pass p.
      __syncthreads();
      if (node < nl && tid == 0) {
        int64_t sum = 0;
        for (int h = 0; h < H; ++h) sum += bcur[h];
        __hip_atomic_store(&xsum[par * kTreeMax + node], ((int64_t)(pass + 1) << 48) | sum,
                           __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (wave == 0) {
        int64_t v = 0;
        int spins = 0;
        while (true) {
          if (lane < nl)
            v = __hip_atomic_load(&xsum[par * kTreeMax + lane], __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
          if (__ballot(lane < nl && (v >> 48) != (int64_t)(pass + 1)) == 0) break;
          __builtin_amdgcn_s_sleep(1);
          if (++spins > (1 << 22)) {  // a member never published: give up, report
            if (lane == 0 && g.status) *g.status = CERTKV_EHIP;
            break;
          }
        }
        if (lane < nl) tsum[lane] = v & (((int64_t)1 << 48) - 1);
      }
      __syncthreads();
      int nd = 0, last = -1;
      for (int j = 0; j < lv; ++j) {
        if (tsum[nd] > B_real) {
          lo = tlam[nd];
          nd = 2 * nd + 2;
        } else {
          hi = tlam[nd];
          last = nd;
          nd = 2 * nd + 1;
        }
      }
      if (node == 0 && last >= 0 && tid < H)
        arg_hi = __hip_atomic_load(&xarg[(par * kTreeMax + last) * 64 + tid], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
      have_bhi = have_bhi || last >= 0;
      __syncthreads();  // every thread has walked the tree before tid 0 rebuilds it
      t += lv;
      ++pass;
    }
    if (node != 0) return;
    if (have_bhi && tid < H) bhi[tid] = arg_hi;
    __syncthreads();
    if (!have_bhi) evaluate(hi, bhi);
  }
  const uint64_t t_bisect = wall_clock64();
  // A head whose curve holds no comparable value from b_min on (all NaN) has
  // no argmin: it starts the repair from b_min.
  if (tid < H && (bhi[tid] < bmin || bhi[tid] > n - 1)) bhi[tid] = bmin;
  __syncthreads();

  int64_t sum0 = 0;
  for (int h = 0; h < H; ++h) sum0 += bhi[h];
  const int64_t R = B_real - sum0;
  const int64_t nrep = R >= 0 ? R : -R;
  const int kmax = (n - 2) / kBlk;  // last block holding an increment i <= n-2

  // Number of increments of head h whose key P is < p (le = false) or <= p
  // (le = true); computed by the 32 threads of half-wave `slot` (< kHeadGroup),
  // which keeps the last curve block it scanned in LDS: once the search has
  // narrowed, successive thresholds cross in the same block and the count
  // reads no global memory.
  auto count_head = [&](int h, double p, bool le, int slot) -> int64_t {
    const int s = bhi[h];
    if (s > n - 2) return 0;
    const int ks = s / kBlk;
    auto crosses = [&](double v) { return le ? (v > p) : (v >= p); };
    const double* ph = pbm + h * nblk;
    int lo_k;  // first block whose running max crosses p
    const int key = rkey[slot];
    const int kc = (key >> 16) == h ? (key & 0xffff) : -1;
    if (kc >= ks && kc <= kmax && crosses(ph[kc]) && (kc == ks || !crosses(ph[kc - 1]))) {
      lo_k = kc;
    } else {
      lo_k = ks;
      int hi_k = kmax + 1;
      while (lo_k < hi_k) {
        const int mid = (lo_k + hi_k) >> 1;
        if (crosses(ph[mid])) hi_k = mid;
        else lo_k = mid + 1;
      }
    }
    if (lo_k > kmax) return (int64_t)(n - 1 - s);
    float* rc = rcache + slot * kRcStride;  // c(lo_k kBlk + i), i = 0..kBlk
    if (lo_k != kc) {
      const float* ch = curves + lht_base(g, l, h, tok0);
      float v[(kBlk + 32) / 32];
#pragma unroll
      for (int m = 0; m < (kBlk + 32) / 32; ++m) {
        const int i = sub + 32 * m;
        v[m] = i <= kBlk ? cval(ch[min(lo_k * kBlk + i, n - 1)]) : 0.f;
      }
#pragma unroll
      for (int m = 0; m < (kBlk + 32) / 32; ++m) {
        const int i = sub + 32 * m;
        if (i <= kBlk) rc[i] = v[m];
      }
      // every thread of the half-wave has read rkey above; the block is read
      // back by other threads of the same wave
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if (sub == 0) rkey[slot] = (h << 16) | lo_k;
    }
    const int i0 = max(lo_k * kBlk, s), i1 = min(lo_k * kBlk + kBlk - 1, n - 2);
    int first = 0x7fffffff;
#pragma unroll
    for (int m = kBlk / 32 - 1; m >= 0; --m) {
      const int r = sub + 32 * m, i = lo_k * kBlk + r;
      const double d = (double)rc[r + 1] - (double)rc[r];
      if (i >= i0 && i <= i1 && crosses(d)) first = i;
    }
    first = half_min_i32(first);
    return (int64_t)(first - s);
  };
  auto total_count = [&](double p, bool le, int64_t* per_head) -> int64_t {
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        const int64_t c = count_head(h, p, le, hg);
        if (sub == 0) per_head[h] = c;
      }
    }
    __syncthreads();
    int64_t tot = 0;
    for (int h = 0; h < H; ++h) tot += per_head[h];
    __syncthreads();
    return tot;
  };

  if (R > 0 && fast) {
    // pbm[h*nblk + k] = running max of d_h over [s_h, end of block k] for the
    // blocks k >= block of s_h (s_h = bhi[h]); -inf before it.  The block
    // maxima come into LDS with all threads; each head's running maximum is
    // then a prefix maximum over its blocks by one half-wave (a run of
    // blocks per thread, then a scan of the runs).
    for (int i = tid; i < H * nblk; i += kAllocThreads) {
      const int h = i / nblk, k = i - h * nblk;
      pbm[i] = dmax[unit_index(g, l, b, h) * nblk_max + k];
    }
    if (tid < kHeadGroup) rkey[tid] = -1;
    __syncthreads();
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        const float* ch = curves + lht_base(g, l, h, tok0);
        const int s = bhi[h];
        const int ks = s / kBlk;
        double dm = -INFINITY;
        if (s <= n - 2) {
          const int e1 = min(ks * kBlk + kBlk - 1, n - 2);
          for (int i = s + sub; i <= e1; i += 32)
            dm = fmax(dm, (double)cval(ch[i + 1]) - (double)cval(ch[i]));
        }
#pragma unroll
        for (int m = 16; m >= 1; m >>= 1) dm = fmax(dm, __shfl_xor(dm, m, 64));
        // block values: the partial first block, then the block maxima up to
        // the last block holding an increment; -inf elsewhere
        double* ph = pbm + h * nblk;
        const bool none = s > n - 2;
        auto val = [&](int k) -> double {
          if (none || k < ks) return -INFINITY;
          if (k == ks) return dm;
          return k <= kmax ? ph[k] : -INFINITY;
        };
        const int per = (nblk + 31) / 32;
        const int k0 = sub * per, k1 = min(nblk, k0 + per);
        double run = -INFINITY;
        for (int k = k0; k < k1; ++k) run = fmax(run, val(k));
        // exclusive prefix maximum of the runs over the half-wave
        double incl = run;
#pragma unroll
        for (int off = 1; off < 32; off <<= 1) {
          const double y = __shfl_up(incl, off, 32);
          if (sub >= off) incl = fmax(incl, y);
        }
        double acc = __shfl_up(incl, 1, 32);
        if (sub == 0) acc = -INFINITY;
        // each thread reads and rewrites only its own blocks, each block's
        // value read just before it is overwritten
        for (int k = k0; k < k1; ++k) {
          acc = fmax(acc, val(k));
          ph[k] = (none || k < ks) ? -INFINITY : acc;
        }
      }
    }
    __syncthreads();
    // smallest key x in [-inf, +inf] with count(P <= x) >= R, by a (J+1)-ary
    // search over the ordered bit patterns (count(P <= +inf) covers every
    // increment): each step counts at J interior points of [klo, khi) at once,
    // one half-wave per (point, head).
    uint64_t klo = dkey(-INFINITY), khi = dkey(INFINITY);
    // A = 2^la <= kHeadGroup / H (at least 2) parts per step, so that the
    // points need no division; (point, head) pairs beyond the half-waves
    // (more than 32 heads) are taken in further rounds
    int la = 1;
    while ((2 << la) <= kHeadGroup / H) ++la;
    const int J = (1 << la) - 1;
    // interior point j: klo + floor(span (j+1) / 2^la), < khi, without overflow
    auto point = [&](uint64_t lo_k, uint64_t span, int j) -> uint64_t {
      return lo_k + (span >> la) * (uint64_t)(j + 1) +
             (((span & (uint64_t)J) * (uint64_t)(j + 1)) >> la);
    };
    while (klo < khi) {
      const uint64_t span = khi - klo;
      for (int gi = hg; gi < J * H; gi += kHeadGroup) {
        const int j = gi / H, h = gi - j * H;
        const int64_t c = count_head(h, dval(point(klo, span, j)), true, hg);
        if (sub == 0) cnt_j[gi] = c;
      }
      __syncthreads();
      // first point whose count reaches R (the counts grow with the point):
      // lane j of wave 0 totals point j over the heads
      if (wave == 0) {
        int64_t c = 0;
        if (lane < J)
          for (int h = 0; h < H; ++h) c += cnt_j[lane * H + h];
        const uint64_t reach = __ballot(lane < J && c >= R);
        if (lane == 0) sfirst = reach ? (int)__builtin_ctzll(reach) : J;
      }
      __syncthreads();
      const int first = sfirst;
      if (first < J) {
        const uint64_t nlo = first > 0 ? point(klo, span, first - 1) + 1 : klo;
        khi = point(klo, span, first);
        klo = nlo;
      } else {
        klo = point(klo, span, J - 1) + 1;
      }
    }
    const double pstar = dval(klo);
    total_count(pstar, false, cnt_lt);
    total_count(pstar, true, cnt_le);
    if (tid == 0) {
      int64_t rem = R;
      for (int h = 0; h < H; ++h) rem -= cnt_lt[h];
      for (int h = 0; h < H; ++h) {
        const int64_t eq = cnt_le[h] - cnt_lt[h];
        const int64_t take = rem < eq ? rem : eq;
        rem -= take;
        bhi[h] = bhi[h] + (int32_t)(cnt_lt[h] + take);
      }
    }
    __syncthreads();
    if (tid < H) budgets[unit_index(g, l, b, tid)] = bhi[tid];
  } else if (tid < 64) {
    // Sequential repair (large problems, or the unreachable removal case).
    const bool act = lane < H;
    int bh = act ? bhi[lane] : 0;
    const float* ch = act ? curves + lht_base(g, l, lane, tok0) : curves;
    int64_t sum = sum0;
    int wbase = bh;  // win[lane][i] = c(wbase + i)
    if (act)
      for (int i = 0; i <= kRepairWin && wbase + i < n; ++i) win[lane][i] = cval(ch[wbase + i]);
    while (sum < B_real) {
      double d = INFINITY;
      if (act && bh < n - 1) {
        if (bh + 1 - wbase > kRepairWin) {
          wbase = bh;
          for (int i = 0; i <= kRepairWin && wbase + i < n; ++i) win[lane][i] = cval(ch[wbase + i]);
        }
        d = (double)win[lane][bh + 1 - wbase] - (double)win[lane][bh - wbase];
      }
      const BestFB r = wave_lexmin(d, act ? lane : 0x7fffffff);
      if (r.f == INFINITY) break;  // unreachable: B_real <= H (n - 1)
      if (lane == r.b) ++bh;
      ++sum;
    }
    while (sum > B_real) {
      double d = INFINITY;
      if (act && bh > bmin) d = (double)cval(ch[bh - 1]) - (double)cval(ch[bh]);
      const BestFB r = wave_lexmin(d, act ? lane : 0x7fffffff);
      if (r.f == INFINITY) break;  // unreachable: H b_min <= B_real
      if (lane == r.b) --bh;
      --sum;
    }
    if (act) budgets[unit_index(g, l, b, lane)] = bh;
  }
  if (stats && tid == 0) {
    stats[((int64_t)l * g.B + b) * 3 + 0] = nrep;
    stats[((int64_t)l * g.B + b) * 3 + 1] = (int64_t)(t_bisect - t_start);
    stats[((int64_t)l * g.B + b) * 3 + 2] = (int64_t)(wall_clock64() - t_bisect);
  }
}

certkv_status run_allocate(const AllocArgs& a, const SeqTab& st, hipStream_t s) {
  // Workgroups per (layer, sequence): a node tree of 3 or 7 when every group
  // of the launch then still has a compute unit per workgroup (one
  // allocation workgroup fills a compute unit's LDS), else 1.
  const int groups = st.count * a.g.L;
  int K = 1;
  if (a.sync && a.steps > 1 && groups <= kSyncGroups) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return CERTKV_EHIP;
    const int cus = device_cus(dev);
    K = 7 * groups <= cus ? 7 : 3 * groups <= cus ? 3 : 1;
  }
  const int per_unit = (a.nblk_max + 4 * kBsBlocks - 1) / (4 * kBsBlocks);
  CERTKV_LAUNCH("curve_blockstats", curve_blockstats_kernel, dim3(a.g.H * st.count * per_unit, a.g.L),
                dim3(256), 0, s, a.g, st, a.nblk_max, a.curves, a.cmin, a.cmaxb, a.cpos, a.dmax,
                K > 1 ? a.sync : (int32_t*)nullptr, (int32_t)kSyncArg);
  if (K > 1) {
    CERTKV_LAUNCH("allocate", allocate_kernel, dim3((unsigned)(K * groups)), dim3(kAllocThreads), 0,
                  s, a.g, st, a.curves, (const float*)a.cmin, (const float*)a.cmaxb,
                  (const int32_t*)a.cpos, (const double*)a.dmax, a.nblk_max, a.steps, a.budgets,
                  a.repairs, K, a.sync);
  } else {
    CERTKV_LAUNCH("allocate", allocate_kernel, dim3(st.count, a.g.L), dim3(kAllocThreads), 0, s,
                  a.g, st, a.curves, (const float*)a.cmin, (const float*)a.cmaxb,
                  (const int32_t*)a.cpos, (const double*)a.dmax, a.nblk_max, a.steps, a.budgets,
                  a.repairs, 1, (int32_t*)nullptr);
  }
  return CERTKV_OK;
}

}  // namespace certkv
