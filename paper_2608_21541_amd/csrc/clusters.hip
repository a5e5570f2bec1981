// Clustered tail summaries on gfx950.
//
// The deterministic output-error bound for clustered tail summaries (appendix)
// stores, per head, m summaries of the evicted tail instead of one slot: for
// each group of the evicted ranks its count n_g, a representative key kbar_g
// and value vbar_g, and radii R_g >= |k_j - kbar_g|, rho_g >= |v_j - vbar_g|
// over its members.  Here the groups are m contiguous runs of the evicted
// ranks b..n-1 in the pass's order (score descending), ceil((n - b) / m)
// ranks each; the representatives are the unweighted means (fp64 sums,
// stored in the cache dtype) and the radii are measured against the stored
// representatives in fp64 and rounded up to fp32, so they hold for what a
// decode reads.  The workgroup of group 0 also records the largest kept value
// norm, one of the terms of the runtime certificate.
//
// One 256-thread workgroup per (unit, group): a pass over the members sums
// keys and values (a thread per (tensor, dim), rows four at a time), then a
// pass measures the distances (a wave per row, lanes over dims).
#include "stages.h"

namespace certkv {

constexpr int kClThreads = 256;

template <typename T>
__device__ __forceinline__ float cl_load(const T* p);
template <>
__device__ __forceinline__ float cl_load<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <>
__device__ __forceinline__ float cl_load<float>(const float* p) { return *p; }

template <typename T>
__device__ __forceinline__ T cl_store(float x);
template <>
__device__ __forceinline__ uint16_t cl_store<uint16_t>(float x) { return f32_to_bf16_rne(x); }
template <>
__device__ __forceinline__ float cl_store<float>(float x) { return x; }

// fp32 at or above x (x >= 0)
__device__ __forceinline__ float cl_round_up(double x) {
  float f = (float)x;
  if ((double)f < x) f = __uint_as_float(__float_as_uint(f) + 1u);
  return f;
}

__device__ __forceinline__ double cl_wave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

template <int D, typename T>
__global__ __launch_bounds__(kClThreads) void cluster_tail_kernel(
    Geo g, SeqTab st, int32_t m, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ budgets, const T* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, const T* __restrict__ vc, int64_t v_sl, int64_t v_st, int64_t v_sh,
    T* __restrict__ kbar, T* __restrict__ vbar, int32_t* __restrict__ count,
    float* __restrict__ rk, float* __restrict__ rv, float* __restrict__ vmax_kept) {
  __shared__ double rep[2][D];
  __shared__ double wmax[3][kClThreads / 64];
  const int gi = blockIdx.x % m;
  const int hb = blockIdx.x / m;
  const int h = hb % g.H, bi = hb / g.H, l = blockIdx.y;
  const int n = st.len[bi];
  const int64_t tok0 = st.start[bi];
  const int64_t u = unit_index(g, l, st.first + bi, h);
  const int64_t base = lht_base(g, l, h, tok0);
  const int b = budgets[u];
  const int E = n - b;
  const int cs = (E + m - 1) / m;
  const int r0 = min(n, b + gi * cs), r1 = min(n, r0 + cs);
  const int cnt = r1 - r0;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const T* kh = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;
  const T* vh = vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh;
  const int64_t cu = u * m + gi;
  // pass 1: sums over the members, thread t -> tensor t / D, dim t % D
  if (t < 2 * D) {
    const int kv = t / D, dd = t % D;
    const T* x = kv ? vh : kh;
    const int64_t xs = kv ? v_st : k_st;
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    int r = r0;
    for (; r + 3 < r1; r += 4) {
      const int j0 = perm[base + r], j1 = perm[base + r + 1];
      const int j2 = perm[base + r + 2], j3 = perm[base + r + 3];
      s0 += (double)cl_load(x + (int64_t)j0 * xs + dd);
      s1 += (double)cl_load(x + (int64_t)j1 * xs + dd);
      s2 += (double)cl_load(x + (int64_t)j2 * xs + dd);
      s3 += (double)cl_load(x + (int64_t)j3 * xs + dd);
    }
    for (; r < r1; ++r) s0 += (double)cl_load(x + (int64_t)perm[base + r] * xs + dd);
    const double mean = cnt > 0 ? ((s0 + s1) + (s2 + s3)) / (double)cnt : 0.0;
    const T stored = cl_store<T>((float)mean);
    (kv ? vbar : kbar)[cu * D + dd] = stored;
    rep[kv][dd] = (double)cl_load(&stored);
  }
  __syncthreads();
  // pass 2: squared distances to the stored representatives, a wave per row
  double mk = 0.0, mv = 0.0;
  for (int r = r0 + wave; r < r1; r += kClThreads / 64) {
    const int j = perm[base + r];
    double sk = 0.0, sv = 0.0;
#pragma unroll
    for (int dd = lane; dd < D; dd += 64) {
      const double dk = (double)cl_load(kh + (int64_t)j * k_st + dd) - rep[0][dd];
      const double dv = (double)cl_load(vh + (int64_t)j * v_st + dd) - rep[1][dd];
      sk = fma(dk, dk, sk);
      sv = fma(dv, dv, sv);
    }
    mk = fmax(mk, cl_wave_sum(sk));
    mv = fmax(mv, cl_wave_sum(sv));
  }
  // group 0 also takes the largest kept value norm (ranks 0..b-1)
  double mkept = 0.0;
  if (gi == 0) {
    for (int r = wave; r < b; r += kClThreads / 64) {
      const int j = perm[base + r];
      double sv = 0.0;
#pragma unroll
      for (int dd = lane; dd < D; dd += 64) {
        const double x = (double)cl_load(vh + (int64_t)j * v_st + dd);
        sv = fma(x, x, sv);
      }
      mkept = fmax(mkept, cl_wave_sum(sv));
    }
  }
  if (lane == 0) {
    wmax[0][wave] = mk;
    wmax[1][wave] = mv;
    wmax[2][wave] = mkept;
  }
  __syncthreads();
  if (t == 0) {
    double a = 0.0, c = 0.0, e = 0.0;
    for (int w = 0; w < kClThreads / 64; ++w) {
      a = fmax(a, wmax[0][w]);
      c = fmax(c, wmax[1][w]);
      e = fmax(e, wmax[2][w]);
    }
    count[cu] = cnt;
    rk[cu] = cl_round_up(sqrt(a));
    rv[cu] = cl_round_up(sqrt(c));
    if (gi == 0) vmax_kept[u] = cl_round_up(sqrt(e));
  }
}

template <int D, typename T>
static certkv_status launch_clusters(const ClusterArgs& a, const SeqTab& st, hipStream_t s) {
  const Geo& g = a.g;
  const dim3 grid((unsigned)(g.H * st.count * a.m), (unsigned)g.L);
  CERTKV_LAUNCH("cluster_tail", (cluster_tail_kernel<D, T>), grid, dim3(kClThreads), 0, s, g, st,
                a.m, a.perm, a.budgets, static_cast<const T*>(a.k.ptr), a.k.s_layer, a.k.s_token,
                a.k.s_head, static_cast<const T*>(a.v.ptr), a.v.s_layer, a.v.s_token, a.v.s_head,
                static_cast<T*>(a.kbar), static_cast<T*>(a.vbar), a.count, a.rk, a.rv,
                a.vmax_kept);
  return CERTKV_OK;
}

certkv_status run_clusters(const ClusterArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.dtype == CERTKV_BF16)
    return a.g.D == 128 ? launch_clusters<128, uint16_t>(a, st, s)
                        : launch_clusters<64, uint16_t>(a, st, s);
  return a.g.D == 128 ? launch_clusters<128, float>(a, st, s) : launch_clusters<64, float>(a, st, s);
}

}  // namespace certkv
