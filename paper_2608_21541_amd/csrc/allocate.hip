// Budget allocation (multiplier bisection + one-token repair) on gfx950.
//
// One workgroup per (layer, sequence).  Each bisection step needs, for every
// head, the smallest b in [b_min, n-1] minimizing f(b) = fma(lambda, b, c(b))
// in fp64 on the fp32 curve.  Scanning all H*n candidates 40 times would
// re-read the curves from L2 40 times, so the scan is pruned exactly:
// for a block of 256 ranks starting at b0 (clamped to b_min) with block
// minimum cmin, every candidate b >= b0 has lambda*b + c(b) >= lambda*b0 +
// cmin, and round-to-nearest is monotone, so LB = fma(lambda, b0, cmin) <=
// f(b) for the whole block.  A block whose (LB, b0) is lexicographically above
// the current best (f*, b*) cannot hold the answer (ties favour smaller b), so
// only the block with the smallest LB and the blocks whose LB undercuts the
// best found in it are evaluated candidate by candidate.  The result is
// identical to the full scan.
//
// Repair runs on one wave, lane h owning head h, with each head's next curve
// values cached in LDS.
#include "stages.h"

namespace certkv {

constexpr int kAllocThreads = 256;
constexpr int kHeadGroup = 8;     // heads evaluated concurrently (32 threads each)
constexpr int kBlk = 256;         // ranks per pruning block
constexpr int kRepairWin = 64;    // cached curve values per head during repair

struct BestFB {
  double f;
  int b;
};

__device__ __forceinline__ bool lex_less(double f1, int b1, double f2, int b2) {
  return f1 < f2 || (f1 == f2 && b1 < b2);
}

// Lexicographic (f, b) minimum over the 32 lanes of a half-wave.
__device__ __forceinline__ BestFB half_wave_min(double f, int b) {
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) {
    double fo = __shfl_xor(f, m, 64);
    int bo = __shfl_xor(b, m, 64);
    if (lex_less(fo, bo, f, b)) {
      f = fo;
      b = bo;
    }
  }
  return BestFB{f, b};
}

// argmin_b fma(lam, b, c(b)) over [bmin, n-1] for one head, by the 32 threads
// with sub = 0..31.  Returns the same value in all 32 threads.
__device__ int head_argmin(const float* __restrict__ ch, const float* __restrict__ mh, int n,
                           int bmin, double lam, int sub) {
  const int nblk = (n + kBlk - 1) / kBlk;
  const int kfirst = bmin / kBlk;
  // (a) block with the smallest lower bound
  double lbest = INFINITY;
  int kbest = 0x7fffffff;
  for (int k = kfirst + sub; k < nblk; k += 32) {
    const int b0 = max(k * kBlk, bmin);
    const double lb = fma(lam, (double)b0, (double)mh[k]);
    if (lex_less(lb, k, lbest, kbest)) {
      lbest = lb;
      kbest = k;
    }
  }
  BestFB kb = half_wave_min(lbest, kbest);
  const int kstar = kb.b;
  // (b) exact minimum inside that block
  double fbest = INFINITY;
  int bbest = 0x7fffffff;
  {
    const int lo = max(kstar * kBlk, bmin), hi = min(kstar * kBlk + kBlk - 1, n - 1);
    for (int bb = lo + sub; bb <= hi; bb += 32) {
      const double f = fma(lam, (double)bb, (double)ch[bb]);
      if (lex_less(f, bb, fbest, bbest)) {
        fbest = f;
        bbest = bb;
      }
    }
  }
  BestFB fb = half_wave_min(fbest, bbest);
  // (c) every other block whose bound undercuts (f*, b*)
  double f2 = fb.f;
  int b2 = fb.b;
  for (int k = kfirst + sub; k < nblk; k += 32) {
    if (k == kstar) continue;
    const int b0 = max(k * kBlk, bmin);
    const double lb = fma(lam, (double)b0, (double)mh[k]);
    if (lex_less(lb, b0, fb.f, fb.b)) {
      const int hi = min(k * kBlk + kBlk - 1, n - 1);
      for (int bb = b0; bb <= hi; ++bb) {
        const double f = fma(lam, (double)bb, (double)ch[bb]);
        if (lex_less(f, bb, f2, b2)) {
          f2 = f;
          b2 = bb;
        }
      }
    }
  }
  return half_wave_min(f2, b2).b;
}

__global__ __launch_bounds__(kAllocThreads) void allocate_kernel(
    Geo g, SeqTab st, const float* __restrict__ curves, const float* __restrict__ cmin,
    int32_t cmin_stride, const float* __restrict__ cmax, int32_t steps,
    int32_t* __restrict__ budgets, int64_t* __restrict__ repairs) {
  __shared__ int32_t bcur[64];
  __shared__ int32_t bhi[64];
  __shared__ float win[64][kRepairWin + 1];

  const int bl = blockIdx.x;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int64_t B_real = st.b_real[bl];
  const int bmin = st.b_min[bl];
  const int H = g.H;
  const int tid = threadIdx.x;
  const int sub = tid & 31;
  const int hg = tid >> 5;

  double cm = 0.0;
  for (int h = 0; h < H; ++h) cm = fmax(cm, (double)cmax[unit_index(g, l, b, h)]);
  double lo = 0.0, hi = 2.0 * cm + 1.0;

  auto evaluate = [&](double lam, int32_t* out) {
    for (int h0 = 0; h0 < H; h0 += kHeadGroup) {
      const int h = h0 + hg;
      if (h < H) {
        const float* ch = curves + lht_base(g, l, h, tok0);
        const float* mh = cmin + unit_index(g, l, b, h) * cmin_stride;
        const int bh = head_argmin(ch, mh, n, bmin, lam, sub);
        if (sub == 0) out[h] = bh;
      }
    }
  };

  evaluate(hi, bhi);
  __syncthreads();
  for (int t = 0; t < steps; ++t) {
    const double lam = (lo + hi) / 2.0;
    evaluate(lam, bcur);
    __syncthreads();
    int64_t sum = 0;
    for (int h = 0; h < H; ++h) sum += bcur[h];
    if (sum > B_real) {
      lo = lam;
    } else {
      hi = lam;
      if (tid < H) bhi[tid] = bcur[tid];
    }
    __syncthreads();
  }

  // Repair to the exact budget: one wave, lane h = head h.
  if (tid < 64) {
    const int lane = tid;
    const bool act = lane < H;
    int bh = act ? bhi[lane] : 0;
    const float* ch = act ? curves + lht_base(g, l, lane, tok0) : curves;
    int64_t sum = 0;
    for (int h = 0; h < H; ++h) sum += bhi[h];
    int64_t nrep = 0;
    int wbase = bh;  // win[lane][i] = c(wbase + i)
    if (act)
      for (int i = 0; i <= kRepairWin && wbase + i < n; ++i) win[lane][i] = ch[wbase + i];
    while (sum < B_real) {
      double d = INFINITY;
      if (act && bh < n - 1) {
        if (bh + 1 - wbase > kRepairWin) {
          wbase = bh;
          for (int i = 0; i <= kRepairWin && wbase + i < n; ++i) win[lane][i] = ch[wbase + i];
        }
        d = (double)win[lane][bh + 1 - wbase] - (double)win[lane][bh - wbase];
      }
      double dm = d;
      int hm = act ? lane : 0x7fffffff;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        double dof = __shfl_xor(dm, m, 64);
        int ho = __shfl_xor(hm, m, 64);
        if (lex_less(dof, ho, dm, hm)) {
          dm = dof;
          hm = ho;
        }
      }
      if (dm == INFINITY) break;  // unreachable: B_real <= H (n - 1)
      if (lane == hm) ++bh;
      ++sum;
      ++nrep;
    }
    while (sum > B_real) {
      double d = INFINITY;
      if (act && bh > bmin) d = (double)ch[bh - 1] - (double)ch[bh];
      double dm = d;
      int hm = act ? lane : 0x7fffffff;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        double dof = __shfl_xor(dm, m, 64);
        int ho = __shfl_xor(hm, m, 64);
        if (lex_less(dof, ho, dm, hm)) {
          dm = dof;
          hm = ho;
        }
      }
      if (dm == INFINITY) break;  // unreachable: H b_min <= B_real
      if (lane == hm) --bh;
      --sum;
      ++nrep;
    }
    if (act) budgets[unit_index(g, l, b, lane)] = bh;
    if (repairs && lane == 0) repairs[(int64_t)l * g.B + b] = nrep;
  }
}

// Block minima and maximum of caller-supplied curves (the allocation-only path).
__global__ __launch_bounds__(256) void block_minmax_kernel(Geo g, SeqTab st,
                                                            const float* __restrict__ curves,
                                                            float* __restrict__ cmin,
                                                            int32_t cmin_stride,
                                                            float* __restrict__ cmax) {
  __shared__ float wmx[4];
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t u = unit_index(g, l, b, h);
  const float* ch = curves + lht_base(g, l, h, st.start[bl]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float mx = -INFINITY;
  const int nblk = (n + kBlk - 1) / kBlk;
  for (int k = wave; k < nblk; k += 4) {
    float mn = INFINITY;
    for (int i = lane; i < kBlk; i += 64) {
      const int bb = k * kBlk + i;
      if (bb < n) {
        mn = fminf(mn, ch[bb]);
        mx = fmaxf(mx, ch[bb]);
      }
    }
    mn = wave_min_f(mn);
    if (lane == 0) cmin[u * cmin_stride + k] = mn;
  }
  mx = wave_max(mx);
  if (lane == 0) wmx[wave] = mx;
  __syncthreads();
  if (threadIdx.x == 0) cmax[u] = fmaxf(fmaxf(wmx[0], wmx[1]), fmaxf(wmx[2], wmx[3]));
}


certkv_status run_allocate(const AllocArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.need_minmax)
    CERTKV_LAUNCH("curve_block_minmax", block_minmax_kernel, dim3(a.g.H * st.count, a.g.L),
                  dim3(256), 0, s, a.g, st, a.curves, a.cmin, a.cmin_stride, a.cmax);
  CERTKV_LAUNCH("allocate", allocate_kernel, dim3(st.count, a.g.L), dim3(kAllocThreads), 0, s, a.g,
                st, a.curves, (const float*)a.cmin, a.cmin_stride, (const float*)a.cmax, a.steps,
                a.budgets, a.repairs);
  return CERTKV_OK;
}

}  // namespace certkv
