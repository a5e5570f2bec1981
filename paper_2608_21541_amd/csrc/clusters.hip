// Clustered tail summaries on gfx950.
//
// The deterministic output-error bound for clustered tail summaries (appendix)
// stores, per head, m summaries of the evicted tail instead of one slot: for
// each group of the evicted ranks its count n_g, a representative key kbar_g
// and value vbar_g, and radii R_g >= |k_j - kbar_g|, rho_g >= |v_j - vbar_g|
// over its members (the cluster-radii equation asks for no more than these
// inequalities).  Here the groups are m contiguous runs of the evicted ranks
// b..n-1 in the pass's order (score descending), ceil((n - b) / m) ranks
// each; the representatives are the unweighted means (fp64 sums, stored in
// the cache dtype).  The radii come from one pass over the members: with c_g
// the mean of every S-th member, S = n_g / 64 clamped to [1, 16] (a
// provisional centre, computed first from that sample), R_g = max_j
// |k_j - c_g| + |c_g - kbar_g| by the
// triangle inequality, likewise rho_g, in fp64 and rounded up to fp32, so
// they hold for the stored representatives a decode reads.  The workgroups
// of a unit also share out its kept ranks for the largest kept value norm,
// one of the terms of the runtime certificate.
//
// One 256-thread workgroup per (unit, group); D/8 lanes take the key slice of
// a row and D/8 its value slice (16-byte loads of 8 dims), 256 / (D/4) rows
// per step: the sample's sums, then the members' sums and squared distances
// to the centres (the rows of the next kClRing steps in flight while a step
// is computed), the lane partials reduced over the row groups of a wave by
// shuffles and over the waves in a fixed order through LDS.
#include "stages.h"

namespace certkv {

constexpr int kClThreads = 256;
constexpr int kClSample = 16;  // largest member stride of the provisional centre's sample
constexpr int kClRing = 4;     // row slices in flight per lane

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

// The raw 8 elements of a row slice (16 bytes of bf16, 32 of fp32), loaded
// as a whole and unpacked when used.
template <typename T>
struct Raw8 {
  uint4 w[sizeof(T) / 2];
};
template <typename T>
__device__ __forceinline__ void cl_raw8(const T* p, Raw8<T>& r) {
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 2); ++i) r.w[i] = reinterpret_cast<const uint4*>(p)[i];
}
template <typename T>
__device__ __forceinline__ void cl_unpack8(const Raw8<T>& r, float* x) {
  if constexpr (sizeof(T) == 2) {
    const uint32_t w[4] = {r.w[0].x, r.w[0].y, r.w[0].z, r.w[0].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf16_lo(w[i]);
      x[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
    const uint32_t w[8] = {r.w[0].x, r.w[0].y, r.w[0].z, r.w[0].w,
                           r.w[1].x, r.w[1].y, r.w[1].z, r.w[1].w};
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __uint_as_float(w[i]);
  }
}

template <int D, typename T>
__global__ __launch_bounds__(kClThreads) void cluster_tail_kernel(
    Geo g, SeqTab st, int32_t m, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ budgets, const T* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, const T* __restrict__ vc, int64_t v_sl, int64_t v_st, int64_t v_sh,
    T* __restrict__ kbar, T* __restrict__ vbar, int32_t* __restrict__ count,
    float* __restrict__ rk, float* __restrict__ rv, float* __restrict__ vmax_kept) {
  constexpr int CL = D / 8;                 // lanes per row slice (8 dims each)
  constexpr int RL = kClThreads / (2 * CL); // rows per step (a K slice and a V slice each)
  constexpr int NW = kClThreads / 64;
  __shared__ double part[NW][2][D];         // per-wave sums
  __shared__ __align__(16) double cen[2][D];  // the sampled centres
  __shared__ double wred[3][NW];
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
  // lane roles: dims 8 cl .. 8 cl + 7 of tensor ts (0 K, 1 V) of rows rl,
  // rl + RL, ...; the 2 CL lanes of a row are consecutive, K slice first
  const int cl = t % CL, ts = (t / CL) & 1, rl = t / (2 * CL);
  const T* xh = ts ? vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh + 8 * cl
                   : kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh + 8 * cl;
  const int64_t x_st = ts ? v_st : k_st;
  const int64_t cu = u * m + gi;

  // Sums of the lane's 8 dims over the rows of the workgroup, in a fixed
  // order: the row groups of a wave by shuffles, then the waves through LDS;
  // thread t < 2 D gets the total of (tensor t / D, dim t % D).
  auto block_sums = [&](double (&sx)[8]) -> double {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int o = 2 * CL; o < 64; o <<= 1) sx[i] += __shfl_xor(sx[i], o, 64);
    }
    if (lane < 2 * CL) {
#pragma unroll
      for (int i = 0; i < 8; ++i) part[wave][ts][8 * cl + i] = sx[i];
    }
    __syncthreads();
    double tot = 0.0;
    if (t < 2 * D)
      for (int w = 0; w < NW; ++w) tot += part[w][t / D][t % D];
    __syncthreads();
    return tot;
  };

  // 1. provisional centres: the mean of members r0, r0 + S, r0 + 2 S, ...
  // with S = cnt / 64 clamped to [1, kClSample] (at least 64 members, or all)
  const int S = min(kClSample, max(1, cnt / 64));
  const int ns = (cnt + S - 1) / S;
  {
    double sx[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) sx[i] = 0.0;
    // kClRing sample rows per lane at a time: their positions, then the rows
    for (int i0 = rl; i0 < ns; i0 += kClRing * RL) {
      int32_t j[kClRing];
#pragma unroll
      for (int q = 0; q < kClRing; ++q) j[q] = perm[base + r0 + min(i0 + q * RL, ns - 1) * S];
      Raw8<T> raw[kClRing];
#pragma unroll
      for (int q = 0; q < kClRing; ++q) cl_raw8(xh + (int64_t)j[q] * x_st, raw[q]);
#pragma unroll
      for (int q = 0; q < kClRing; ++q) {
        float x[8];
        cl_unpack8(raw[q], x);
        const double w = i0 + q * RL < ns ? 1.0 : 0.0;
#pragma unroll
        for (int e = 0; e < 8; ++e) sx[e] = fma(w, (double)x[e], sx[e]);
      }
    }
    const double tot = block_sums(sx);
    if (t < 2 * D) cen[t / D][t % D] = ns > 0 ? tot / (double)ns : 0.0;
    __syncthreads();
  }
  // the lane's centre dims stay in LDS, read per row
  const double2* c2 = reinterpret_cast<const double2*>(&cen[ts][8 * cl]);

  // 2. one pass over the members: sums and squared distances to the centres.
  // One row slice per lane and step; kClRing buffers rotate, each refilled
  // kClRing steps ahead right after it is consumed, the positions of a refill
  // loaded with the refill before it.  Rows past the group are clamped to
  // its last row (always in bounds): such a row adds with weight zero to the
  // sums and repeats a distance already counted.
  double sx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) sx[i] = 0.0;
  double mx = 0.0;
  const int steps = (cnt + RL - 1) / RL;
  auto pos = [&](int r) -> int32_t { return perm[base + min(r, r1 - 1)]; };
  auto consume = [&](const Raw8<T>& raw, int r) {
    float x[8];
    cl_unpack8(raw, x);
    const double w = r < r1 ? 1.0 : 0.0;
    double dd = 0.0;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      const double2 c = c2[i / 2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const double p = (double)x[i + e];
        sx[i + e] = fma(w, p, sx[i + e]);
        const double a = p - (e ? c.y : c.x);
        dd = fma(a, a, dd);
      }
    }
    // the CL lanes of a row slice are consecutive lanes of one wave (every
    // lane runs the same number of steps, so the shuffles stay within full
    // slices)
#pragma unroll
    for (int o = CL / 2; o >= 1; o >>= 1) dd += __shfl_xor(dd, o, 64);
    mx = fmax(mx, dd);
  };
  if (steps > 0) {
    Raw8<T> buf[kClRing];
    int32_t jn[kClRing];
    int32_t j0[kClRing];
#pragma unroll
    for (int q = 0; q < kClRing; ++q) j0[q] = pos(r0 + rl + q * RL);
    // the first fills in the order of the refills below (buffer q, then its
    // next position), so that the count of loads issued after each buffer
    // is the same on entry as around the loop
#pragma unroll
    for (int q = 0; q < kClRing; ++q) {
      cl_raw8(xh + (int64_t)j0[q] * x_st, buf[q]);
      jn[q] = pos(r0 + rl + (q + kClRing) * RL);
      __builtin_amdgcn_sched_barrier(0);
    }
    // No branch in the loop body (so that the compiler's load counting keeps
    // the ring in flight): steps past the group consume clamped rows with
    // weight zero, and the last refills load clamped rows that are never used.
    for (int k = 0; k < steps; k += kClRing) {
#pragma unroll
      for (int q = 0; q < kClRing; ++q) {
        const int r = r0 + rl + (k + q) * RL;
        consume(buf[q], r);
        cl_raw8(xh + (int64_t)jn[q] * x_st, buf[q]);
        jn[q] = pos(r + 2 * kClRing * RL);
        // keep the refill here, kClRing - 1 consumes ahead of its use
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // representatives: the means, as stored
  const double tot = block_sums(sx);
  double e2 = 0.0;  // (c - stored mean)^2 of this thread's (tensor, dim)
  if (t < 2 * D) {
    const int kv = t / D, dd = t % D;
    const double mean = cnt > 0 ? tot / (double)cnt : 0.0;
    const T stored = cl_store<T>((float)mean);
    (kv ? vbar : kbar)[cu * D + dd] = stored;
    const double dc = cen[kv][dd] - (double)cl_load(&stored);
    e2 = dc * dc;
  }
  // The largest kept value norm (ranks 0..b-1): the workgroup of group gi
  // takes the gi-th of m shares of the kept ranks (every lane on value
  // slices, 2 RL rows per step, kClRing steps' rows loaded together) and
  // folds its maximum into vmax_kept[u] below.
  double mkept = 0.0;
  {
    const T* vh = vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh + 8 * cl;
    const int rk2 = t / CL;
    const int kq = (b + m - 1) / m, k0 = min(b, gi * kq), k1 = min(b, k0 + kq);
    for (int i0 = k0 + rk2; i0 < k1; i0 += kClRing * 2 * RL) {
      int32_t j[kClRing];
#pragma unroll
      for (int q = 0; q < kClRing; ++q) j[q] = perm[base + min(i0 + q * 2 * RL, k1 - 1)];
      Raw8<T> raw[kClRing];
#pragma unroll
      for (int q = 0; q < kClRing; ++q) cl_raw8(vh + (int64_t)j[q] * v_st, raw[q]);
#pragma unroll
      for (int q = 0; q < kClRing; ++q) {
        float xv[8];
        cl_unpack8(raw[q], xv);
        double s2 = 0.0;
#pragma unroll
        for (int i = 0; i < 8; ++i) s2 = fma((double)xv[i], (double)xv[i], s2);
#pragma unroll
        for (int o = CL / 2; o >= 1; o >>= 1) s2 += __shfl_xor(s2, o, 64);
        mkept = fmax(mkept, s2);  // clamped rows repeat a counted one
      }
    }
  }
  // largest squared distance of the wave's K slices and of its V slices
  double mk = ts ? 0.0 : mx, mv = ts ? mx : 0.0;
#pragma unroll
  for (int o = 32; o >= CL; o >>= 1) {
    mk = fmax(mk, __shfl_xor(mk, o, 64));
    mv = fmax(mv, __shfl_xor(mv, o, 64));
    mkept = fmax(mkept, __shfl_xor(mkept, o, 64));
  }
  if (lane == 0) {
    wred[0][wave] = mk;
    wred[1][wave] = mv;
    wred[2][wave] = mkept;
  }
  // |c - kbar|^2 and |c - vbar|^2: threads 0..D-1 hold the key terms,
  // D..2D-1 the value terms (D is a multiple of 64: whole waves), summed
  // per wave and then over the waves in order
  double ew = e2;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ew += __shfl_xor(ew, o, 64);
  if (lane == 0) part[wave][0][0] = ew;
  __syncthreads();
  if (t == 0) {
    double a = 0.0, c = 0.0, e = 0.0, ek = 0.0, ev = 0.0;
    for (int w = 0; w < NW; ++w) {
      a = fmax(a, wred[0][w]);
      c = fmax(c, wred[1][w]);
      e = fmax(e, wred[2][w]);
    }
    for (int w = 0; w < D / 64; ++w) ek += part[w][0][0];
    for (int w = D / 64; w < 2 * D / 64; ++w) ev += part[w][0][0];
    count[cu] = cnt;
    rk[cu] = cl_round_up(sqrt(a) + sqrt(ek));
    rv[cu] = cl_round_up(sqrt(c) + sqrt(ev));
    // non-negative floats order as their bit patterns: the maximum over the
    // unit's groups by an integer atomic maximum (vmax_kept cleared first)
    if (e > 0.0) atomicMax(reinterpret_cast<unsigned int*>(vmax_kept + u),
                           __float_as_uint(cl_round_up(sqrt(e))));
  }
}

__global__ void cl_clear_kernel(float* __restrict__ x, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = 0.f;
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

certkv_status run_clusters_clear(float* vmax_kept, int64_t U, hipStream_t s) {
  CERTKV_LAUNCH("cluster_clear", cl_clear_kernel, dim3((unsigned)((U + 255) / 256)), dim3(256), 0,
                s, vmax_kept, U);
  return CERTKV_OK;
}

certkv_status run_clusters(const ClusterArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.dtype == CERTKV_BF16)
    return a.g.D == 128 ? launch_clusters<128, uint16_t>(a, st, s)
                        : launch_clusters<64, uint16_t>(a, st, s);
  return a.g.D == 128 ? launch_clusters<128, float>(a, st, s) : launch_clusters<64, float>(a, st, s);
}

}  // namespace certkv
