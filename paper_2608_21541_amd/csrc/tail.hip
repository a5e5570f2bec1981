// Tail-summary slot and packed-cache compaction.
//
// Per unit the evicted set E is the complement of the kept positions.  The
// slot is the (s)_+-weighted key and value centroid of E; the weights'
// normalizer cancels, so
//   k* = sum_E s_j k_j / sum_E s_j,  v* likewise,  m = sum_E s_j / sum_j s_j.
// When the totals sum_j s_j k_j and sum_j s_j v_j are already known (from the
// scoring and curve kernels) the evicted sums are total minus kept, so only
// the kept rows (about a tenth) are read.  If the evicted mass is below 1/64
// of the total, the evicted rows are summed directly instead (cancellation
// guard; rare).
//
// gather    (nsplit workgroups per unit) copies a slice of the unit's kept
//           rows into the packed cache and forms fp64 partial weighted sums;
// mass      (standalone path only) partial total / evicted score mass;
// finalize  (one workgroup per unit) adds the partials in split order,
//           forms k*, v*, m and appends the slot row.
#include "stages.h"

namespace certkv {

constexpr int kTailThreads = 256;
constexpr double kComplementMinMass = 1.0 / 64.0;

template <typename T>
__device__ __forceinline__ float elem_f32(const uint4& q, int e);
template <>
__device__ __forceinline__ float elem_f32<uint16_t>(const uint4& q, int e) {
  const uint32_t w = (&q.x)[e >> 1];
  return (e & 1) ? bf16_hi(w) : bf16_lo(w);
}
template <>
__device__ __forceinline__ float elem_f32<float>(const uint4& q, int e) {
  return __uint_as_float((&q.x)[e]);
}

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f32_to_bf16_rne(x); }
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }

__device__ __forceinline__ bool is_kept(const uint64_t* bmu, int j) {
  return (bmu[j >> 6] >> (j & 63)) & 1ull;
}

// Clear the per-unit kept bitmaps, then set one bit per kept position.
__global__ void bitmap_clear_kernel(uint64_t* __restrict__ bm, int64_t words) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < words) bm[i] = 0ull;
}

__global__ void bitmap_set_kernel(Geo g, SeqTab st, const int64_t* __restrict__ kept_offsets,
                                  const int32_t* __restrict__ kept_idx, uint64_t* __restrict__ bm,
                                  int32_t bm_stride) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int n = st.len[bl];
  const int64_t u = unit_index(g, l, st.first + bl, h);
  const int64_t o0 = kept_offsets[u], o1 = kept_offsets[u + 1];
  for (int64_t i = o0 + threadIdx.x; i < o1; i += blockDim.x) {
    const int j = kept_idx[i];
    if (j >= 0 && j < n)
      atomicOr(reinterpret_cast<unsigned long long*>(&bm[u * bm_stride + (j >> 6)]),
               1ull << (j & 63));
  }
}

// Partial total and evicted (s)_+ mass over a slice of positions.
__global__ __launch_bounds__(kTailThreads) void mass_kernel(Geo g, SeqTab st, int32_t nsplit,
                                                            const float* __restrict__ scores,
                                                            const uint64_t* __restrict__ bm,
                                                            int32_t bm_stride,
                                                            double* __restrict__ mpart) {
  __shared__ double red[3][kTailThreads / 64];
  const int split = blockIdx.x % nsplit;
  const int hb = blockIdx.x / nsplit;
  const int h = hb % g.H;
  const int bl = hb / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int n = st.len[bl];
  const int64_t u = unit_index(g, l, st.first + bl, h);
  const int64_t sbase = lht_base(g, l, h, st.start[bl]);
  const uint64_t* bmu = bm + u * bm_stride;
  const int per = (n + nsplit - 1) / nsplit;
  const int j0 = split * per, j1 = min(n, j0 + per);
  double sa = 0.0, se = 0.0, ne = 0.0;
  for (int j = j0 + threadIdx.x; j < j1; j += kTailThreads) {
    const float s = scores[sbase + j];
    const double sp = s > 0.f ? (double)s : 0.0;
    sa += sp;
    if (!is_kept(bmu, j)) {
      se += sp;
      ne += 1.0;
    }
  }
  sa = wave_sum(sa);
  se = wave_sum(se);
  ne = wave_sum(ne);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = sa;
    red[1][wave] = se;
    red[2][wave] = ne;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int i = threadIdx.x;
    mpart[(u * nsplit + split) * 3 + i] = red[i][0] + red[i][1] + red[i][2] + red[i][3];
  }
}

// Copy a slice of kept rows to the packed cache and/or accumulate the fp64
// partial weighted key and value sums of the slice.
template <int D, typename T, bool DO_TAIL, bool DO_COMPACT>
__global__ __launch_bounds__(kTailThreads) void tail_gather_kernel(
    Geo g, SeqTab st, int32_t nsplit, const float* __restrict__ scores, const T* __restrict__ kc,
    int64_t k_sl, int64_t k_st, int64_t k_sh, const T* __restrict__ vc, int64_t v_sl,
    int64_t v_st, int64_t v_sh, const int64_t* __restrict__ kept_offsets,
    const int32_t* __restrict__ kept_idx, double* __restrict__ kpart_out,
    T* __restrict__ k_packed, T* __restrict__ v_packed, int32_t* __restrict__ pos_packed) {
  constexpr int EPL = 16 / sizeof(T);      // elements per 16-byte lane chunk
  constexpr int LPR = D / EPL;             // lanes per row
  constexpr int RPS = kTailThreads / LPR;  // rows per workgroup step
  __shared__ double redk[DO_TAIL ? RPS : 1][D];
  __shared__ double redv[DO_TAIL ? RPS : 1][D];

  const int split = blockIdx.x % nsplit;
  const int hb = blockIdx.x / nsplit;
  const int h = hb % g.H;
  const int bl = hb / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int64_t sbase = lht_base(g, l, h, tok0);
  const int64_t u = unit_index(g, l, b, h);
  const int tid = threadIdx.x;
  const int ri = tid / LPR, ci = tid % LPR;
  const int64_t off = kept_offsets[u];
  const int nk = (int)(kept_offsets[u + 1] - off);
  const int per = (nk + nsplit - 1) / nsplit;
  const int i0 = split * per, i1 = min(nk, i0 + per);
  const int64_t poff = off + g.slot * u;  // packed segment start
  const T* kb = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;
  const T* vb = vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh;

  double ak[EPL], av[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) ak[e] = av[e] = 0.0;
  // Four rows per lane group per step: their indices, then their rows and
  // scores, are loaded together so that each step waits for two round trips.
  constexpr int UR = 4;
  for (int i = i0 + ri; i < i1; i += RPS * UR) {
    // The entries past the run read a clamped one and fetch its row again,
    // unused: no load sits behind a branch, so none waits for itself.
    int j[UR];
#pragma unroll
    for (int q = 0; q < UR; ++q)
      j[q] = min(max(kept_idx[off + min(i + q * RPS, i1 - 1)], 0), n - 1);  // caller indices clamped
    uint4 kq[UR], vq[UR];
    float sv[UR];
#pragma unroll
    for (int q = 0; q < UR; ++q) {
      kq[q] = *reinterpret_cast<const uint4*>(kb + (int64_t)j[q] * k_st + ci * EPL);
      vq[q] = *reinterpret_cast<const uint4*>(vb + (int64_t)j[q] * v_st + ci * EPL);
      sv[q] = DO_TAIL ? scores[sbase + j[q]] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < UR; ++q) {
      if (i + q * RPS >= i1) continue;
      const int ii = i + q * RPS;
      if (DO_COMPACT) {
        *reinterpret_cast<uint4*>(k_packed + (poff + ii) * D + ci * EPL) = kq[q];
        *reinterpret_cast<uint4*>(v_packed + (poff + ii) * D + ci * EPL) = vq[q];
        if (ci == 0) pos_packed[poff + ii] = j[q];
      }
      if (DO_TAIL) {
        const double w = sv[q] > 0.f ? (double)sv[q] : 0.0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          ak[e] = fma(w, (double)elem_f32<T>(kq[q], e), ak[e]);
          av[e] = fma(w, (double)elem_f32<T>(vq[q], e), av[e]);
        }
      }
    }
  }
  if (DO_TAIL) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      redk[ri][ci * EPL + e] = ak[e];
      redv[ri][ci * EPL + e] = av[e];
    }
    __syncthreads();
    for (int d = tid; d < D; d += kTailThreads) {
      double sk = 0.0, sv = 0.0;
      for (int r = 0; r < RPS; ++r) {
        sk += redk[r][d];
        sv += redv[r][d];
      }
      kpart_out[((u * nsplit + split) * 2 + 0) * D + d] = sk;
      kpart_out[((u * nsplit + split) * 2 + 1) * D + d] = sv;
    }
  }
}

// Per unit: combine partials, form the slot, append it to the packed cache.
template <int D, typename T, bool DO_TAIL, bool DO_COMPACT>
__global__ __launch_bounds__(kTailThreads) void tail_finalize_kernel(
    Geo g, SeqTab st, int32_t nsplit, const float* __restrict__ scores, const T* __restrict__ kc,
    int64_t k_sl, int64_t k_st, int64_t k_sh, const T* __restrict__ vc, int64_t v_sl,
    int64_t v_st, int64_t v_sh, const int64_t* __restrict__ kept_offsets,
    const uint64_t* __restrict__ bm, int32_t bm_stride, const double* __restrict__ kpart,
    const double* __restrict__ mpart, const double* __restrict__ evicted_sum,
    const double* __restrict__ total_sum, const double* __restrict__ ksum,
    const double* __restrict__ vsum, float* __restrict__ k_star, float* __restrict__ v_star,
    double* __restrict__ tail_mass, T* __restrict__ k_packed, T* __restrict__ v_packed,
    int32_t* __restrict__ pos_packed) {
  constexpr int EPL = 16 / sizeof(T);
  constexpr int LPR = D / EPL;
  constexpr int RPS = kTailThreads / LPR;
  __shared__ double redk[DO_TAIL ? RPS : 1][D];
  __shared__ double redv[DO_TAIL ? RPS : 1][D];
  __shared__ float slot_k[D], slot_v[D];

  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int64_t sbase = lht_base(g, l, h, tok0);
  const int64_t u = unit_index(g, l, b, h);
  const int tid = threadIdx.x;
  const int64_t off = kept_offsets[u];
  const int nk = (int)(kept_offsets[u + 1] - off);

  if (DO_TAIL) {
    double S_all, S_E, nE;
    if (evicted_sum && total_sum) {
      S_all = total_sum[u];
      S_E = evicted_sum[u];
      nE = (double)(n - nk);
    } else {
      S_all = S_E = nE = 0.0;
#pragma unroll 8
      for (int sp = 0; sp < nsplit; ++sp) {
        S_all += mpart[(u * nsplit + sp) * 3 + 0];
        S_E += mpart[(u * nsplit + sp) * 3 + 1];
        nE += mpart[(u * nsplit + sp) * 3 + 2];
      }
    }
    const bool uniform = !(S_all > 0.0);  // every score zero: uniform weights
    if (uniform) {
      S_all = (double)n;
      S_E = nE;
    }
    const bool direct = uniform || !(ksum && vsum) || S_E < kComplementMinMass * S_all;
    if (!direct) {
      for (int d = tid; d < D; d += kTailThreads) {
        double sk = 0.0, sv = 0.0;
        // partials added in split order; unrolled so that the loads of 16
        // splits are in flight together
#pragma unroll 16
        for (int sp = 0; sp < nsplit; ++sp) {
          sk += kpart[((u * nsplit + sp) * 2 + 0) * D + d];
          sv += kpart[((u * nsplit + sp) * 2 + 1) * D + d];
        }
        slot_k[d] = S_E > 0.0 ? (float)((ksum[u * D + d] - sk) / S_E) : 0.f;
        slot_v[d] = S_E > 0.0 ? (float)((vsum[u * D + d] - sv) / S_E) : 0.f;
      }
    } else {
      // Direct weighted sums over the evicted rows of this unit.
      const int ri = tid / LPR, ci = tid % LPR;
      const T* kb = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;
      const T* vb = vc + (int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh;
      const uint64_t* bmu = bm + u * bm_stride;
      double ak[EPL], av[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) ak[e] = av[e] = 0.0;
      for (int j = ri; j < n; j += RPS) {
        if (is_kept(bmu, j)) continue;
        const float s = scores[sbase + j];
        const double w = uniform ? 1.0 : (s > 0.f ? (double)s : 0.0);
        if (w == 0.0) continue;
        const uint4 kq = *reinterpret_cast<const uint4*>(kb + (int64_t)j * k_st + ci * EPL);
        const uint4 vq = *reinterpret_cast<const uint4*>(vb + (int64_t)j * v_st + ci * EPL);
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          ak[e] = fma(w, (double)elem_f32<T>(kq, e), ak[e]);
          av[e] = fma(w, (double)elem_f32<T>(vq, e), av[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        redk[ri][ci * EPL + e] = ak[e];
        redv[ri][ci * EPL + e] = av[e];
      }
      __syncthreads();
      for (int d = tid; d < D; d += kTailThreads) {
        double sk = 0.0, sv = 0.0;
        for (int r = 0; r < RPS; ++r) {
          sk += redk[r][d];
          sv += redv[r][d];
        }
        slot_k[d] = S_E > 0.0 ? (float)(sk / S_E) : 0.f;
        slot_v[d] = S_E > 0.0 ? (float)(sv / S_E) : 0.f;
      }
    }
    __syncthreads();
    for (int d = tid; d < D; d += kTailThreads) {
      k_star[u * D + d] = slot_k[d];
      v_star[u * D + d] = slot_v[d];
    }
    if (tid == 0) tail_mass[u] = S_E / S_all;
  } else {
    for (int d = tid; d < D; d += kTailThreads) {
      slot_k[d] = k_star[u * D + d];
      slot_v[d] = v_star[u * D + d];
    }
    __syncthreads();
  }
  if (DO_COMPACT && g.slot) {
    const int64_t prow = off + u + nk;
    for (int d = tid; d < D; d += kTailThreads) {
      k_packed[prow * D + d] = from_f32<T>(slot_k[d]);
      v_packed[prow * D + d] = from_f32<T>(slot_v[d]);
    }
    if (tid == 0) pos_packed[prow] = -1;
  }
}

template <int D, typename T, bool DT, bool DC>
static certkv_status launch_tail(const TailArgs& a, const SeqTab& st, hipStream_t s) {
  const Geo& g = a.g;
  const dim3 grid_split(g.H * st.count * a.nsplit, g.L);
  const dim3 grid_unit(g.H * st.count, g.L);
  const char* gname = DT ? (DC ? "tail_compact_gather" : "tail_gather") : "compact_gather";
  const char* fname = DT ? (DC ? "tail_compact_finalize" : "tail_finalize") : "compact_slot";
  if (DT && !(a.evicted_sum && a.total_sum))
    CERTKV_LAUNCH("tail_mass", mass_kernel, grid_split, dim3(kTailThreads), 0, s, g, st, a.nsplit,
                  a.scores, (const uint64_t*)a.bitmap, a.bm_stride, a.mpart);
  CERTKV_LAUNCH(gname, (tail_gather_kernel<D, T, DT, DC>), grid_split, dim3(kTailThreads), 0, s, g,
                st, a.nsplit, a.scores, static_cast<const T*>(a.k.ptr), a.k.s_layer, a.k.s_token,
                a.k.s_head, static_cast<const T*>(a.v.ptr), a.v.s_layer, a.v.s_token, a.v.s_head,
                a.kept_offsets, a.kept_idx, a.kpart, static_cast<T*>(a.k_packed),
                static_cast<T*>(a.v_packed), a.pos_packed);
  CERTKV_LAUNCH(fname, (tail_finalize_kernel<D, T, DT, DC>), grid_unit, dim3(kTailThreads), 0, s, g,
                st, a.nsplit, a.scores, static_cast<const T*>(a.k.ptr), a.k.s_layer, a.k.s_token,
                a.k.s_head, static_cast<const T*>(a.v.ptr), a.v.s_layer, a.v.s_token, a.v.s_head,
                a.kept_offsets, (const uint64_t*)a.bitmap, a.bm_stride, (const double*)a.kpart,
                (const double*)a.mpart, a.evicted_sum, a.total_sum, a.ksum, a.vsum, a.k_star,
                a.v_star, a.tail_mass, static_cast<T*>(a.k_packed), static_cast<T*>(a.v_packed),
                a.pos_packed);
  return CERTKV_OK;
}

template <int D, typename T>
static certkv_status dispatch_tail(const TailArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.do_tail && a.do_compact) return launch_tail<D, T, true, true>(a, st, s);
  if (a.do_tail) return launch_tail<D, T, true, false>(a, st, s);
  return launch_tail<D, T, false, true>(a, st, s);
}

certkv_status run_bitmap(const TailArgs& a, const SeqTab& st, int64_t words_total, bool clear,
                         hipStream_t s) {
  if (clear)
    CERTKV_LAUNCH("kept_bitmap_clear", bitmap_clear_kernel, dim3((unsigned)((words_total + 255) / 256)),
                  dim3(256), 0, s, a.bitmap, words_total);
  CERTKV_LAUNCH("kept_bitmap_set", bitmap_set_kernel, dim3(a.g.H * st.count, a.g.L), dim3(256), 0, s,
                a.g, st, a.kept_offsets, a.kept_idx, a.bitmap, a.bm_stride);
  return CERTKV_OK;
}

certkv_status run_tail(const TailArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.dtype == CERTKV_BF16)
    return a.g.D == 128 ? dispatch_tail<128, uint16_t>(a, st, s) : dispatch_tail<64, uint16_t>(a, st, s);
  return a.g.D == 128 ? dispatch_tail<128, float>(a, st, s) : dispatch_tail<64, float>(a, st, s);
}

}  // namespace certkv
