// Dispersion curves c(b) = sqrt((m Q - |W|^2)_+) over the evicted suffix of
// the score order (the keys at ranks b..n-1), for b = 0..n-1, in fp64, with
// m, W and Q the suffix sums of a, a v and a |v|^2.
//
// One workgroup (16 waves) per unit walks the ranks from the top (rank n-1)
// down in chunks of 512.  Wave w owns the 32 ranks [512k + 32(15-w),
// 512k + 32(16-w)) of chunk k and lane i owns dims DP*i..DP*i+DP-1
// (DP = d/64).  Per chunk:
//   phase 1  each wave forms the totals of its 16 rows: m, W (per dim) and
//            Q (sum of a |v|^2);
//   carry    wave w starts from the chunk carry plus the totals of waves
//            0..w-1 (higher ranks), added in that fixed order (deterministic);
//   phase 2  the wave walks its ranks top-down extending m, W and the
//            lane-local part q of Q; per rank each lane forms
//            x = m q - |W|^2 over its dims (lane 0's q starts from Q_carry,
//            the part of Q above the wave) and a
//            transpose-reduce over the 64 lanes, folded in as the ranks are
//            produced, yields c^2 of all 32 ranks.  The last wave's final
//            state is the carry of the next chunk.
// The gathers are software-pipelined: while chunk k is computed, the value
// rows of chunk k-1 are in flight and the order/score entries of chunk k-2
// are being fetched.  Also emitted: sum_j (s_j)_+ v_j (the value total of the
// tail summary).
#include "stages.h"

namespace certkv {

constexpr int kCurveThreads = 1024;
constexpr int kCurveWaves = kCurveThreads / 64;
constexpr int kRPW = 32;                          // ranks per wave and chunk
constexpr int kLev = kRPW == 32 ? 5 : (kRPW == 16 ? 4 : 3);  // log2(kRPW)
constexpr int kCurveChunk = kCurveWaves * kRPW;   // 512 ranks

template <int DP, bool BF16>
__device__ __forceinline__ void unpack_dims(uint32_t raw0, uint32_t raw1, float (&v)[DP]) {
  if (BF16) {
    if (DP == 2) {
      v[0] = bf16_lo(raw0);
      v[DP - 1] = bf16_hi(raw0);
    } else {
      v[0] = bf16_lo(raw0);
    }
  } else {
    v[0] = __uint_as_float(raw0);
    if (DP == 2) v[DP - 1] = __uint_as_float(raw1);
  }
}

// One transpose-reduce step over lane bit 5 (half = true) or 4: lanes with
// the bit clear end with lo + partner's lo, lanes with it set with hi +
// partner's hi.  v_permlane32_swap exchanges the upper half-wave of its first
// operand with the lower half-wave of its second (v_permlane16_swap likewise
// for odd and even rows of 16), which is exactly that exchange.
__device__ __forceinline__ double combine_swap(double lo, double hi, bool half) {
  const uint64_t a = (uint64_t)__double_as_longlong(lo);
  const uint64_t b = (uint64_t)__double_as_longlong(hi);
  uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32), b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
  if (half) {
    const auto r0 = __builtin_amdgcn_permlane32_swap(a0, b0, false, false);
    const auto r1 = __builtin_amdgcn_permlane32_swap(a1, b1, false, false);
    a0 = r0[0]; b0 = r0[1]; a1 = r1[0]; b1 = r1[1];
  } else {
    const auto r0 = __builtin_amdgcn_permlane16_swap(a0, b0, false, false);
    const auto r1 = __builtin_amdgcn_permlane16_swap(a1, b1, false, false);
    a0 = r0[0]; b0 = r0[1]; a1 = r1[0]; b1 = r1[1];
  }
  const double x = __longlong_as_double((long long)(((uint64_t)a1 << 32) | a0));
  const double y = __longlong_as_double((long long)(((uint64_t)b1 << 32) | b0));
  return x + y;
}

template <int D, bool BF16>
__global__ __launch_bounds__(kCurveThreads) void curves_kernel(
    Geo g, SeqTab st, const uint32_t* __restrict__ sorted_keys, const int32_t* __restrict__ perm,
    const double* __restrict__ ssum, const void* __restrict__ vc, int64_t v_sl, int64_t v_st,
    int64_t v_sh, float* __restrict__ curves, double* __restrict__ vsum) {
  constexpr int DP = D / 64;
  constexpr int RAW = (BF16 || DP == 1) ? 1 : 2;  // 32-bit words per lane per row
  __shared__ double tW[kCurveWaves][D];   // phase-1 totals per wave
  __shared__ double tQ[kCurveWaves];
  __shared__ double tM[kCurveWaves];
  // chunk carry (suffix sums above the chunk), double-buffered by chunk
  // parity: the last wave writes the next carry while others may still read
  // the current one
  __shared__ double cW[2][D];
  __shared__ double cQM[2][2];

  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int64_t base = lht_base(g, l, h, tok0);
  const int64_t u = unit_index(g, l, b, h);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const double tot = ssum[u];
  const double inv_n = 1.0 / (double)n;
  // Value slice of this (layer, head, sequence): rows of d elements, token
  // stride v_st; the host guarantees it spans less than 4 GiB.
  constexpr int E = BF16 ? 2 : 4;
  const BufRsrc vrs = make_rsrc(
      static_cast<const char*>(vc) + ((int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh) * E,
      (uint32_t)(((int64_t)(n - 1) * v_st + D) * E));
  const uint32_t vrow_bytes = (uint32_t)(v_st * E);
  const uint32_t vlane = (uint32_t)(lane * DP * E);
  const BufRsrc krs = make_rsrc(sorted_keys + base, (uint32_t)n * 4u);
  const BufRsrc prs = make_rsrc(perm + base, (uint32_t)n * 4u);

  // rank of lane r (< kRPW) of this wave in chunk k; lane 0 = highest rank
  auto rank_of = [&](int k, int r) {
    return k * kCurveChunk + (kCurveWaves - 1 - wave) * kRPW + kRPW - 1 - r;
  };
  // Order entry and radix key of lane r of chunk k.  Every lane loads (from a
  // clamped, in-bounds rank) so that no branch splits the pipelined loads;
  // `valid` marks the lanes that hold a real rank of this wave.  The weight
  // is formed one iteration later, when the loads have landed.
  auto fetch_meta = [&](int k, uint32_t& key, int& pos, bool& valid) {
    const int rk = rank_of(k, lane);
    valid = k >= 0 && lane < kRPW && rk < n;
    const uint32_t idx = (uint32_t)min(max(rk, 0), n - 1) * 4u;
    key = buf_load_u32(krs, idx);
    pos = (int)buf_load_u32(prs, idx);
  };
  // weight a = (s)_+ / sum (s)_+ (uniform when every score is zero); zero for
  // absent ranks, whose rows then add nothing
  auto weight = [&](uint32_t key, bool valid) -> double {
    if (!valid) return 0.0;
    const float s = desc_key_value(key);
    return tot > 0.0 ? (s > 0.f ? (double)s / tot : 0.0) : inv_n;
  };
  auto row_of = [&](int pos, bool valid) { return valid ? min(max(pos, 0), n - 1) : 0; };
  // Value rows of the 32 ranks of chunk k (row 0 stands in for absent ranks,
  // whose weight is zero).
  auto fetch_rows = [&](int pos, uint32_t (&raw)[kRPW][RAW]) {
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      // the row offset is uniform (scalar offset of the load); rows are
      // clamped into the sequence, so soff + vlane stays inside the slice
      const int pr = __builtin_amdgcn_readlane(pos, r);
      const uint32_t soff = (uint32_t)pr * vrow_bytes;
      if (RAW == 2) {
        const uint2 w2 = buf_load_u64s(vrs, vlane, soff);
        raw[r][0] = w2.x;
        raw[r][RAW - 1] = w2.y;
      } else if (BF16 && DP == 1) {
        raw[r][0] = buf_load_u16s(vrs, vlane, soff);
      } else {
        raw[r][0] = buf_load_u32s(vrs, vlane, soff);
      }
    }
  };

  const int nch = (n + kCurveChunk - 1) / kCurveChunk;
  for (int i = threadIdx.x; i < D; i += kCurveThreads) cW[(nch - 1) & 1][i] = 0.0;
  if (threadIdx.x < 2) cQM[(nch - 1) & 1][threadIdx.x] = 0.0;

  double a_cur, a_n1;
  int p_cur, p_n1, p_n2;
  uint32_t k_cur, k_n1, k_n2;
  bool ok_cur, ok_n1, ok_n2;
  uint32_t vcur[kRPW][RAW], vnext[kRPW][RAW];
  fetch_meta(nch - 1, k_cur, p_cur, ok_cur);
  fetch_meta(nch - 2, k_n1, p_n1, ok_n1);
  a_cur = weight(k_cur, ok_cur);
  a_n1 = weight(k_n1, ok_n1);
  p_cur = row_of(p_cur, ok_cur);
  p_n1 = row_of(p_n1, ok_n1);
  fetch_rows(p_cur, vcur);

  for (int k = nch - 1; k >= 0; --k) {
    // pipeline: order entries two chunks ahead, value rows one chunk ahead
    fetch_meta(k - 2, k_n2, p_n2, ok_n2);
    fetch_rows(p_n1, vnext);

    // weight of lane r's rank, as a wave-uniform (scalar) value
    auto a_at = [&](int r) -> double {
      const uint64_t u = (uint64_t)__double_as_longlong(a_cur);
      const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, r);
      const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), r);
      return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
    };

    // phase 1: totals of the wave's rows
    {
      double sW[DP], sQ = 0.0, sM = 0.0;
#pragma unroll
      for (int t = 0; t < DP; ++t) sW[t] = 0.0;
#pragma unroll
      for (int r = 0; r < kRPW; ++r) {
        const double ar = a_at(r);
        float v[DP];
        unpack_dims<DP, BF16>(vcur[r][0], vcur[r][RAW - 1], v);
        double vv = 0.0;
#pragma unroll
        for (int t = 0; t < DP; ++t) {
          const double vd = (double)v[t];
          sW[t] = fma(ar, vd, sW[t]);
          vv = fma(vd, vd, vv);
        }
        sQ = fma(ar, vv, sQ);
        sM += ar;
      }
      sQ = wave_sum(sQ);
#pragma unroll
      for (int t = 0; t < DP; ++t) tW[wave][lane * DP + t] = sW[t];
      if (lane == 0) {
        tQ[wave] = sQ;
        tM[wave] = sM;
      }
    }
    __syncthreads();
    // carry of this wave: chunk carry + totals of the waves above it
    const int par = k & 1;
    double W[DP], m = cQM[par][1], Qc = cQM[par][0];
#pragma unroll
    for (int t = 0; t < DP; ++t) W[t] = cW[par][lane * DP + t];
    for (int w2 = 0; w2 < wave; ++w2) {
#pragma unroll
      for (int t = 0; t < DP; ++t) W[t] += tW[w2][lane * DP + t];
      Qc += tQ[w2];
      m += tM[w2];
    }
    // Opaque to the optimizer: keeps the rows packed between the phases
    // instead of holding their converted doubles.
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      __asm__ volatile("" : "+v"(vcur[r][0]));
      if (RAW == 2) __asm__ volatile("" : "+v"(vcur[r][RAW - 1]));
    }
    // phase 2: walk the ranks top-down.  Streaming transpose-reduce of the
    // per-lane values over lane bits 5, 4, ...: ranks 2i and 2i+1 combine over
    // lane bit 5 as soon as both exist, pairs of those over bit 4, and so on,
    // so at most one pending value per level is live.  Lane bit 5 - j ends up
    // naming rank bit j.
    // lane 0 carries the chunk's Q above the wave, so that every lane forms
    // m * q - |W|^2 over its dims and their sum is m Q - |W|^2
    double q = lane == 0 ? Qc : 0.0;
    double pend[kLev];
    double c2 = 0.0;
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const double ar = a_at(r);
      float v[DP];
      unpack_dims<DP, BF16>(vcur[r][0], vcur[r][RAW - 1], v);
      double vv = 0.0, w2 = 0.0;
#pragma unroll
      for (int t = 0; t < DP; ++t) {
        const double vd = (double)v[t];
        W[t] = fma(ar, vd, W[t]);
        w2 = fma(W[t], W[t], w2);
        vv = fma(vd, vd, vv);
      }
      m += ar;
      q = fma(ar, vv, q);
      double cur = fma(m, q, -w2);
      bool placed = false;
#pragma unroll
      for (int lev = 0; lev < kLev; ++lev) {
        if (placed) continue;
        if (((r >> lev) & 1) == 0) {
          pend[lev] = cur;
          placed = true;
        } else if (lev < 2) {
          cur = combine_swap(pend[lev], cur, lev == 0);
        } else {
          const int msk = 32 >> lev;
          const bool up = (lane & msk) != 0;
          const double keep = up ? cur : pend[lev];
          const double send = up ? pend[lev] : cur;
          cur = keep + __shfl_xor(send, msk, 64);
        }
      }
      if (!placed) c2 = cur;
    }
    // the lanes sharing a rank: add their copies
#pragma unroll
    for (int m2 = 1; m2 < 64 / kRPW; m2 <<= 1) c2 += __shfl_xor(c2, m2, 64);
    int r_mine = 0;
#pragma unroll
    for (int lev = 0; lev < kLev; ++lev) r_mine |= ((lane >> (5 - lev)) & 1) << lev;
    const int rk = rank_of(k, r_mine);
    if ((lane & (64 / kRPW - 1)) == 0 && rk < n) {
      if (!isfinite(c2)) report_nonfinite(g);
      curves[base + rk] = (float)sqrt(c2 > 0.0 ? c2 : 0.0);
    }
    // the last wave's final state carries into the next chunk
    if (wave == kCurveWaves - 1) {
#pragma unroll
      for (int t = 0; t < DP; ++t) cW[par ^ 1][lane * DP + t] = W[t];
      if (lane == 0) {
        cQM[par ^ 1][0] = Qc + tQ[wave];
        cQM[par ^ 1][1] = m;
      }
    }
    __syncthreads();
    // rotate the pipeline
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      vcur[r][0] = vnext[r][0];
      if (RAW == 2) vcur[r][RAW - 1] = vnext[r][RAW - 1];
    }
    a_cur = a_n1;
    a_n1 = weight(k_n2, ok_n2);
    p_n1 = row_of(p_n2, ok_n2);
  }
  if (vsum && wave == 0) {
#pragma unroll
    for (int t = 0; t < DP; ++t) vsum[u * D + lane * DP + t] = cW[1][lane * DP + t] * tot;
  }
}

certkv_status run_curves(const CurveArgs& a, const SeqTab& st, hipStream_t s) {
  dim3 grid(a.g.H * st.count, a.g.L);
  if (a.dtype == CERTKV_BF16) {
    if (a.g.D == 128)
      CERTKV_LAUNCH("curves", (curves_kernel<128, true>), grid, dim3(kCurveThreads), 0, s, a.g, st,
                    a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,
                    a.curves, a.vsum);
    else
      CERTKV_LAUNCH("curves", (curves_kernel<64, true>), grid, dim3(kCurveThreads), 0, s, a.g, st,
                    a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,
                    a.curves, a.vsum);
  } else {
    if (a.g.D == 128)
      CERTKV_LAUNCH("curves", (curves_kernel<128, false>), grid, dim3(kCurveThreads), 0, s, a.g, st,
                    a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,
                    a.curves, a.vsum);
    else
      CERTKV_LAUNCH("curves", (curves_kernel<64, false>), grid, dim3(kCurveThreads), 0, s, a.g, st,
                    a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,
                    a.curves, a.vsum);
  }
  return CERTKV_OK;
}

}  // namespace certkv
