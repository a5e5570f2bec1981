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
// One 256-thread workgroup per (unit, group), D/8 lanes per row (16-byte
// loads of 8 dims of K and V) and 256 / (D/8) rows in flight: a pass over
// the members sums keys and values in fp64 (row-lane partials combined in a
// fixed order through LDS), then a pass measures the distances (reduced over
// the lanes of a row by shuffles).
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

// Eight consecutive elements of a row as floats (16 bytes of bf16, or 32 of
// fp32).
template <typename T>
__device__ __forceinline__ void cl_load8(const T* p, float* x);
template <>
__device__ __forceinline__ void cl_load8<uint16_t>(const uint16_t* p, float* x) {
  const uint4 r = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = bf16_lo(w[i]);
    x[2 * i + 1] = bf16_hi(w[i]);
  }
}
template <>
__device__ __forceinline__ void cl_load8<float>(const float* p, float* x) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 c = reinterpret_cast<const float4*>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
}

template <int D, typename T>
__global__ __launch_bounds__(kClThreads) void cluster_tail_kernel(
    Geo g, SeqTab st, int32_t m, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ budgets, const T* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, const T* __restrict__ vc, int64_t v_sl, int64_t v_st, int64_t v_sh,
    T* __restrict__ kbar, T* __restrict__ vbar, int32_t* __restrict__ count,
    float* __restrict__ rk, float* __restrict__ rv, float* __restrict__ vmax_kept) {
  constexpr int CL = D / 8;                 // lanes per row (8 dims each)
  constexpr int RL = kClThreads / CL;       // rows in flight
  __shared__ double part[RL][2][D];         // per row-lane sums, then the representatives
  __shared__ double wmax[3][kClThreads / 64];
  const int gi = blockIdx.x % m;
  const int hb = blockIdx.x / m;
  const int h = hb % g.H, bi = hb / g.H, l = blockIdx.y;
  const int n = st.len[bi];
  const int64_t tok0 = st.start[bi];
  const int64_t u = unit_index(g, l, st.first + bi, h);
  const int64_t base = lht_base(g, l, h, tok0);
  const int b = min(max(budgets[u], 0), n);  // caller budgets clamped into [0, n]
  const int E = n - b;
  const int cs = (E + m - 1) / m;
  const int r0 = min(n, b + gi * cs), r1 = min(n, r0 + cs);
  const int cnt = r1 - r0;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int cl = t % CL, rl = t / CL;       // dims 8 cl .. 8 cl + 7 of rows rl, rl + RL, ...
  const T* kh = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh + 8 * cl;
  const T* vh = vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh + 8 * cl;
  const int64_t cu = u * m + gi;
  // pass 1: sums over the members (fp64), each lane its 8 dims of K and V
  double sk[8], sv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) sk[i] = sv[i] = 0.0;
  // Two rows per lane and step (rows r and r + RL), their positions loaded
  // one step ahead; positions past the group are clamped to its last row
  // (always in bounds) and such a row is added with weight zero.
  const int steps = (cnt + 2 * RL - 1) / (2 * RL);
  int64_t ja = cnt > 0 ? perm[base + min(r0 + rl, r1 - 1)] : 0;
  int64_t jb = cnt > 0 ? perm[base + min(r0 + rl + RL, r1 - 1)] : 0;
  for (int k = 0; k < steps; ++k) {
    const int r = r0 + rl + 2 * k * RL;
    const int64_t j0 = ja, j1 = jb;
    ja = perm[base + min(r + 2 * RL, r1 - 1)];
    jb = perm[base + min(r + 3 * RL, r1 - 1)];
    float xk0[8], xv0[8], xk1[8], xv1[8];
    cl_load8(kh + j0 * k_st, xk0);
    cl_load8(vh + j0 * v_st, xv0);
    cl_load8(kh + j1 * k_st, xk1);
    cl_load8(vh + j1 * v_st, xv1);
    const double w0 = r < r1 ? 1.0 : 0.0, w1 = r + RL < r1 ? 1.0 : 0.0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sk[i] = fma(w0, (double)xk0[i], sk[i]);
      sv[i] = fma(w0, (double)xv0[i], sv[i]);
      sk[i] = fma(w1, (double)xk1[i], sk[i]);
      sv[i] = fma(w1, (double)xv1[i], sv[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    part[rl][0][8 * cl + i] = sk[i];
    part[rl][1][8 * cl + i] = sv[i];
  }
  __syncthreads();
  if (t < 2 * D) {  // one thread per (tensor, dim): the row-lanes' sums in order
    const int kv = t / D, dd = t % D;
    double s = 0.0;
    for (int q = 0; q < RL; ++q) s += part[q][kv][dd];
    const double mean = cnt > 0 ? s / (double)cnt : 0.0;
    const T stored = cl_store<T>((float)mean);
    (kv ? vbar : kbar)[cu * D + dd] = stored;
    sk[0] = (double)cl_load(&stored);
  }
  __syncthreads();
  if (t < 2 * D) part[0][t / D][t % D] = sk[0];
  __syncthreads();
  double rep_k[8], rep_v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    rep_k[i] = part[0][0][8 * cl + i];
    rep_v[i] = part[0][1][8 * cl + i];
  }
  // pass 2: squared distances to the stored representatives; the CL lanes of
  // a row are consecutive lanes of one wave, reduced by shuffles
  // (every lane runs the same number of steps, so the shuffles stay
  // within full row groups)
  // (clamped rows repeat the group's last row, whose distance is counted
  // anyway, so the maximum is unchanged)
  double mk = 0.0, mv = 0.0;
  ja = cnt > 0 ? perm[base + min(r0 + rl, r1 - 1)] : 0;
  jb = cnt > 0 ? perm[base + min(r0 + rl + RL, r1 - 1)] : 0;
  for (int k = 0; k < steps; ++k) {
    const int r = r0 + rl + 2 * k * RL;
    const int64_t j0 = ja, j1 = jb;
    ja = perm[base + min(r + 2 * RL, r1 - 1)];
    jb = perm[base + min(r + 3 * RL, r1 - 1)];
    float xk0[8], xv0[8], xk1[8], xv1[8];
    cl_load8(kh + j0 * k_st, xk0);
    cl_load8(vh + j0 * v_st, xv0);
    cl_load8(kh + j1 * k_st, xk1);
    cl_load8(vh + j1 * v_st, xv1);
    double dk0 = 0.0, dv0 = 0.0, dk1 = 0.0, dv1 = 0.0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const double a0 = (double)xk0[i] - rep_k[i], c0 = (double)xv0[i] - rep_v[i];
      const double a1 = (double)xk1[i] - rep_k[i], c1 = (double)xv1[i] - rep_v[i];
      dk0 = fma(a0, a0, dk0);
      dv0 = fma(c0, c0, dv0);
      dk1 = fma(a1, a1, dk1);
      dv1 = fma(c1, c1, dv1);
    }
#pragma unroll
    for (int o = CL / 2; o >= 1; o >>= 1) {
      dk0 += __shfl_xor(dk0, o, 64);
      dv0 += __shfl_xor(dv0, o, 64);
      dk1 += __shfl_xor(dk1, o, 64);
      dv1 += __shfl_xor(dv1, o, 64);
    }
    mk = fmax(mk, fmax(dk0, dk1));
    mv = fmax(mv, fmax(dv0, dv1));
  }
  // group 0 also takes the largest kept value norm (ranks 0..b-1)
  double mkept = 0.0;
  if (gi == 0) {
    const int ksteps = (b + RL - 1) / RL;
    for (int k = 0; k < ksteps; ++k) {
      const int r = rl + k * RL;
      double s2 = 0.0;
      if (r < b) {
        const int64_t j = perm[base + r];
        float xv[8];
        cl_load8(vh + j * v_st, xv);
#pragma unroll
        for (int i = 0; i < 8; ++i) s2 = fma((double)xv[i], (double)xv[i], s2);
      }
#pragma unroll
      for (int o = CL / 2; o >= 1; o >>= 1) s2 += __shfl_xor(s2, o, 64);
      mkept = fmax(mkept, s2);
    }
  }
#pragma unroll
  for (int o = 32; o >= CL; o >>= 1) {
    mk = fmax(mk, __shfl_xor(mk, o, 64));
    mv = fmax(mv, __shfl_xor(mv, o, 64));
    mkept = fmax(mkept, __shfl_xor(mkept, o, 64));
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
