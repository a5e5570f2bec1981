// Dispersion curves c(b) = sqrt((m Q - |W|^2)_+) over the evicted suffix of
// the score order (the keys at ranks b..n-1), for b = 0..n-1, in fp64.
//
// One workgroup (8 waves) per unit walks the ranks from the top (rank n-1)
// down in chunks of 256.  Wave w owns the 32 ranks
// [256k + 32(7-w), 256k + 32(8-w)) of chunk k and lane i owns dims
// DP*i..DP*i+DP-1 (DP = d/64):
//   phase 1  each wave gathers its 32 value rows (by perm) into VGPRs and
//            forms its totals m, W (per dim) and Q;
//   carry    wave w starts from the chunk carry plus the totals of waves
//            0..w-1 (higher ranks), summed in that fixed order;
//   phase 2  the wave walks its ranks top-down extending m and W and the
//            local part of Q; per rank each lane forms
//              x = m * (local Q of its dims) - |its W dims|^2,
//            lane 0 adds m * Q_carry, and a transpose-reduce over the 64
//            lanes yields c^2 for 16 ranks at a time.
// Besides c (fp32), the kernel emits sum_j (s_j)_+ v_j (the value total of the
// tail summary).
#include "stages.h"

namespace certkv {

constexpr int kCurveThreads = 512;
constexpr int kCurveWaves = kCurveThreads / 64;
constexpr int kRPW = 32;                          // ranks per wave and chunk
constexpr int kCurveChunk = kCurveWaves * kRPW;   // 256 ranks

template <int DP>
__device__ __forceinline__ void unpack_dims(uint32_t raw, float (&v)[DP]) {
  if (DP == 2) {
    v[0] = bf16_lo(raw);
    v[DP - 1] = bf16_hi(raw);
  } else {
    v[0] = bf16_lo(raw);
  }
}

template <int D, bool BF16>
__global__ __launch_bounds__(kCurveThreads) void curves_kernel(
    Geo g, SeqTab st, const uint32_t* __restrict__ sorted_keys, const int32_t* __restrict__ perm,
    const double* __restrict__ ssum, const void* __restrict__ vc, int64_t v_sl, int64_t v_st,
    int64_t v_sh, float* __restrict__ curves, double* __restrict__ vsum) {
  constexpr int DP = D / 64;
  __shared__ double tW[kCurveWaves][D];
  __shared__ double tQ[kCurveWaves];
  __shared__ double tM[kCurveWaves];
  __shared__ double a_lds[kCurveWaves][kRPW];
  __shared__ int32_t pos_lds[kCurveWaves][kRPW];

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

  // chunk carry (identical in every wave)
  double cW[DP], cQ = 0.0, cM = 0.0;
#pragma unroll
  for (int t = 0; t < DP; ++t) cW[t] = 0.0;

  const int nch = (n + kCurveChunk - 1) / kCurveChunk;
  for (int k = nch - 1; k >= 0; --k) {
    const int lo = k * kCurveChunk + (kCurveWaves - 1 - wave) * kRPW;  // lowest rank of wave
    const int rank = lo + kRPW - 1 - lane;  // lane 0 = highest rank of the sub-chunk
    const bool live = lane < kRPW && rank < n;
    // weights a = (s)_+ / sum (s)_+ (uniform when every score is zero)
    double a = 0.0;
    int32_t pos = 0;
    if (live) {
      const float s = desc_key_value(sorted_keys[base + rank]);
      pos = min(max(perm[base + rank], 0), n - 1);
      a = tot > 0.0 ? (s > 0.f ? (double)s / tot : 0.0) : inv_n;
    }
    if (lane < kRPW) {
      a_lds[wave][lane] = a;
      pos_lds[wave][lane] = pos;
    }
    // gather the value rows, lane i holding dims DP*i..
    uint32_t vraw[kRPW];
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const int pr = pos_lds[wave][r];
      const bool lr = (lo + kRPW - 1 - r) < n;
      vraw[r] = 0u;
      if (lr) {
        const int64_t off = (int64_t)l * v_sl + (tok0 + pr) * v_st + (int64_t)h * v_sh + lane * DP;
        if (BF16) {
          const uint16_t* vp = static_cast<const uint16_t*>(vc) + off;
          vraw[r] = DP == 2 ? *reinterpret_cast<const uint32_t*>(vp) : (uint32_t)vp[0];
        } else {
          const float* vp = static_cast<const float*>(vc) + off;
          vraw[r] = __float_as_uint(vp[0]);  // fp32 values: one dim per lane (d = 64)
        }
      }
    }
    // phase 1: sub-chunk totals
    double sW[DP], sP = 0.0, sM = 0.0;
#pragma unroll
    for (int t = 0; t < DP; ++t) sW[t] = 0.0;
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const double ar = a_lds[wave][r];
      float v[DP];
      if (BF16) {
        unpack_dims<DP>(vraw[r], v);
      } else {
        v[0] = __uint_as_float(vraw[r]);
      }
      sM += ar;
#pragma unroll
      for (int t = 0; t < DP; ++t) {
        const double p = ar * (double)v[t];
        sW[t] += p;
        sP += p * (double)v[t];
      }
    }
    sP = wave_sum(sP);
#pragma unroll
    for (int t = 0; t < DP; ++t) tW[wave][lane * DP + t] = sW[t];
    if (lane == 0) {
      tQ[wave] = sP;
      tM[wave] = sM;
    }
    __syncthreads();
    // carry of this wave: chunk carry + totals of the waves above it
    double W[DP], m = cM, Qc = cQ;
#pragma unroll
    for (int t = 0; t < DP; ++t) W[t] = cW[t];
    for (int w2 = 0; w2 < wave; ++w2) {
#pragma unroll
      for (int t = 0; t < DP; ++t) W[t] += tW[w2][lane * DP + t];
      Qc += tQ[w2];
      m += tM[w2];
    }
    // Opaque to the optimizer: keeps the rows packed in 32-bit registers
    // between the phases instead of holding 2*kRPW converted doubles.
#pragma unroll
    for (int r = 0; r < kRPW; ++r) __asm__ volatile("" : "+v"(vraw[r]));
    // phase 2: walk the wave's ranks top-down, 16 at a time
    double PL[DP];
#pragma unroll
    for (int t = 0; t < DP; ++t) PL[t] = 0.0;
#pragma unroll
    for (int q4 = 0; q4 < kRPW / 16; ++q4) {
      double x[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int r = q4 * 16 + j;
        const double ar = a_lds[wave][r];
        float v[DP];
        if (BF16) {
          unpack_dims<DP>(vraw[r], v);
        } else {
          v[0] = __uint_as_float(vraw[r]);
        }
        m += ar;
        double xl = 0.0, pl = 0.0;
#pragma unroll
        for (int t = 0; t < DP; ++t) {
          const double p = ar * (double)v[t];
          W[t] += p;
          PL[t] += p * (double)v[t];
          pl += PL[t];
          xl -= W[t] * W[t];
        }
        xl += m * pl;
        if (lane == 0) xl += m * Qc;
        x[j] = xl;
      }
      // transpose-reduce 16 values over lane bits 5..2, then sum lane bits 1..0
#pragma unroll
      for (int msk = 32, half = 8; msk >= 4; msk >>= 1, half >>= 1) {
        const bool up = (lane & msk) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
          double keep = up ? x[half + i] : x[i];
          double send = up ? x[i] : x[half + i];
          x[i] = keep + __shfl_xor(send, msk, 64);
        }
      }
      double c2 = x[0];
      c2 += __shfl_xor(c2, 1, 64);
      c2 += __shfl_xor(c2, 2, 64);
      // value index held = lane bits 5..2 -> j = lane >> 2 within this group of 16
      const int j = lane >> 2;
      const int rk = lo + kRPW - 1 - (q4 * 16 + j);
      const float c = (float)sqrt(c2 > 0.0 ? c2 : 0.0);
      if ((lane & 3) == 0 && rk < n) curves[base + rk] = c;
    }
    __syncthreads();
    // advance the chunk carry by every wave's totals, in wave order
    for (int w2 = 0; w2 < kCurveWaves; ++w2) {
#pragma unroll
      for (int t = 0; t < DP; ++t) cW[t] += tW[w2][lane * DP + t];
      cQ += tQ[w2];
      cM += tM[w2];
    }
    __syncthreads();
  }
  if (vsum && wave == 0) {
#pragma unroll
    for (int t = 0; t < DP; ++t) vsum[u * D + lane * DP + t] = cW[t] * tot;
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
    if (a.g.D != 64) return CERTKV_EUNSUPPORTED;
    CERTKV_LAUNCH("curves", (curves_kernel<64, false>), grid, dim3(kCurveThreads), 0, s, a.g, st,
                  a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,
                  a.curves, a.vsum);
  }
  return CERTKV_OK;
}

}  // namespace certkv
