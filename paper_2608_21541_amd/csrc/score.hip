// Observation-window scoring on gfx950.
//
// For KV head h the M = w*G window rows (query head g of the group, window
// position q) give logits l = scale * <q_row, k_j>; the score of key j is the
// sum over rows of the row-softmax weight of key j.  Two passes over K:
//   pass 1  per key block: running (max, sum of exp) of every row -> partials
//   combine per row: log-sum-exp over blocks
//   pass 2  per key block: s_j = sum_rows exp(l_row,j - lse_row), written out,
//           plus (optionally) the block's sum_j s_j k_j for the tail summary.
// The contraction runs on MFMA v_mfma_f32_16x16x32_bf16 with key tiles as the
// A operand (rows = 16 keys, held in VGPRs straight from HBM) and the window
// queries as the B operand (columns = 16 queries, staged once per workgroup in
// LDS).  Each lane then owns one query column, so row statistics
// are lane-local and per-key sums are one cross-lane reduction per key tile.
// Exponentials use v_exp_f32 on log2-domain logits.
#include "stages.h"

namespace certkv {

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kScoreThreads = 256;     // 4 waves
constexpr int kKeysPerWaveIter = 64;   // two 32-key tiles per wave
constexpr int kKeysPerIter = 256;      // per workgroup iteration

union Frag {
  uint4 u;
  bf16x8_t v;
};

// LDS row stride of the staged window queries, in bf16 elements (16-byte pad
// against bank conflicts).
template <int D>
struct ScoreSmem {
  static constexpr int kRowElems = D + 8;
};

// MFMA v_mfma_f32_16x16x32_bf16 layout used below (per 64-lane wave):
//   A (16 keys x 32 dims): lane (grp = lane/16, c = lane%16) supplies key c,
//     8 consecutive dims of its group's slice;
//   B (32 dims x 16 queries): the same lane supplies query c, same dims;
//   D (16 x 16): lane (grp, c) holds query column c, key rows 4*grp + r,
//     r = 0..3.
// Each lane group owns a contiguous quarter of the head dimension for all of
// its k-steps, so a lane loads one 2*D/4-byte run of its key row.
constexpr int kNqtMax = 32;  // up to 512 window rows (16 per query tile)

template <int D, bool P2>
__global__ __launch_bounds__(kScoreThreads) void score_mfma_kernel(
    Geo g, SeqTab st, const uint16_t* __restrict__ qw, int64_t q_sl, int64_t q_st,
    int64_t q_sh, const uint16_t* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, int32_t keys_per_block, int32_t nkb_max, float2* __restrict__ part,
    const float* __restrict__ lse2, float* __restrict__ scores,
    float* __restrict__ kpart) {
  constexpr int KS = D / 32;   // MFMA k-steps
  constexpr int QD = D / 4;    // dims per lane group
  constexpr int RE = ScoreSmem<D>::kRowElems;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  uint16_t* q_lds = reinterpret_cast<uint16_t*>(smem_raw);

  const int kb = blockIdx.x;
  const int h = blockIdx.y % g.H;
  const int bl = blockIdx.y / g.H;
  const int l = blockIdx.z;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  const int key_begin = kb * keys_per_block;
  if (key_begin >= n) return;
  const int key_end = min(n, key_begin + keys_per_block);
  const int M = g.w * g.G;
  const int Mp = (M + 15) & ~15;  // rows padded to whole 16-query tiles
  const int64_t u = unit_index(g, l, b, h);

  float* lse_lds = reinterpret_cast<float*>(smem_raw + (size_t)Mp * RE * 2);
  float* red_lds = lse_lds + Mp;  // [4][Mp][2] or [4][D]

  // Stage the window queries of this KV head: row rho = q*G + gq; padding
  // rows are zero and are never written out (pass 2 gives them lse = +inf).
  {
    const int chunks = D / 8;
    for (int c = threadIdx.x; c < Mp * chunks; c += kScoreThreads) {
      int rho = c / chunks, part8 = c % chunks;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (rho < M) {
        int qq = rho / g.G, gq = rho % g.G;
        const uint16_t* src = qw + (int64_t)l * q_sl + (int64_t)(b * g.w + qq) * q_st +
                              (int64_t)(h * g.G + gq) * q_sh + part8 * 8;
        val = *reinterpret_cast<const uint4*>(src);
      }
      *reinterpret_cast<uint4*>(q_lds + rho * RE + part8 * 8) = val;
    }
    if (P2) {
      for (int i = threadIdx.x; i < Mp; i += kScoreThreads)
        lse_lds[i] = i < M ? lse2[u * M + i] : INFINITY;
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = lane >> 4;
  const int c16 = lane & 15;
  const float c2 = g.scale * kLog2e;
  const int nqt = Mp / 16;
  const int first_masked = g.causal ? (n - g.w + 1) : n;  // keys >= this may be masked
  const uint16_t* kbase = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;

  float mrun[kNqtMax], srun[kNqtMax];  // pass 1: this lane's query column, per tile
#pragma unroll
  for (int i = 0; i < kNqtMax; ++i) {
    mrun[i] = -INFINITY;
    srun[i] = 0.f;
  }
  float kacc[QD];  // pass 2: weighted key sum over this lane's dims
#pragma unroll
  for (int i = 0; i < QD; ++i) kacc[i] = 0.f;

  for (int it = key_begin + wave * kKeysPerWaveIter; it < key_end; it += kKeysPerIter) {
    // Four 16-key tiles (keys it..it+63) as A fragments, straight from HBM.
    Frag kf[4][KS];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      int key = it + t * 16 + c16;
      int keyc = key < n ? key : n - 1;
      const uint4* src = reinterpret_cast<const uint4*>(kbase + (int64_t)keyc * k_st + grp * QD);
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[t][s].u = src[s];
    }
    const bool need_mask = (it + 63 >= first_masked) || (it + 63 >= n);
    float ssum[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) ssum[t][r] = 0.f;

#pragma unroll
    for (int qt = 0; qt < kNqtMax; ++qt) {
      if (qt >= nqt) break;
      f32x4_t acc[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const uint16_t* qrow = q_lds + (qt * 16 + c16) * RE + grp * QD;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        Frag qf;
        qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[t][s].v, qf.v, acc[t], 0, 0, 0);
      }
      if (need_mask) {
        const int qpos = n - g.w + (qt * 16 + c16) / g.G;
        const int lim = g.causal ? min(qpos, n - 1) : n - 1;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (it + t * 16 + grp * 4 + r > lim) acc[t][r] = -INFINITY;
      }
      if (!P2) {
        float mx = acc[0][0];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, acc[t][r]);
        const float mnew = fmaxf(mrun[qt], mx * c2);
        if (mnew != -INFINITY) {
          const float sc = __builtin_amdgcn_exp2f(mrun[qt] - mnew);
          float sacc = 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) sacc += __builtin_amdgcn_exp2f(fmaf(acc[t][r], c2, -mnew));
          srun[qt] = fmaf(srun[qt], sc, sacc);
          mrun[qt] = mnew;
        }
      } else {
        const float l2 = lse_lds[qt * 16 + c16];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) ssum[t][r] += __builtin_amdgcn_exp2f(fmaf(acc[t][r], c2, -l2));
      }
    }

    if (P2) {
      // Sum each key's per-lane partials over the 16 query columns of its lane
      // group: transpose-reduce so lane (grp, c16) ends with value index c16,
      // i.e. tile c16/4, register c16%4 = key 16*(c16/4) + 4*grp + c16%4.
      float v[16];
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) v[t * 4 + r] = ssum[t][r];
#pragma unroll
      for (int m = 8, half = 8; m >= 1; m >>= 1, half >>= 1) {
        const bool up = (lane & m) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
          float keep = up ? v[half + i] : v[i];
          float send = up ? v[i] : v[half + i];
          v[i] = keep + __shfl_xor(send, m, 64);
        }
      }
      const float s_mine = v[0];
      const int key_mine = it + (c16 >> 2) * 16 + grp * 4 + (c16 & 3);
      if (key_mine < n) scores[lht_base(g, l, h, tok0) + key_mine] = s_mine;
      if (kpart) {
        // Lane (grp, c16) holds key c16 of each tile over dims grp*QD..; the
        // score of key (t, i) sits in lane 16*(i/4) + 4*t + i%4.
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int src = 16 * (c16 >> 2) + 4 * t + (c16 & 3);
          float s_t = __shfl(s_mine, src, 64);
          const int key = it + t * 16 + c16;
          s_t = (key < n && s_t > 0.f) ? s_t : 0.f;
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            const uint32_t* w4 = reinterpret_cast<const uint32_t*>(&kf[t][s].u);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              kacc[s * 8 + 2 * e] = fmaf(s_t, bf16_lo(w4[e]), kacc[s * 8 + 2 * e]);
              kacc[s * 8 + 2 * e + 1] = fmaf(s_t, bf16_hi(w4[e]), kacc[s * 8 + 2 * e + 1]);
            }
          }
        }
      }
    }
  }

  if (!P2) {
    // Merge the four lane groups (same query column, other key rows), then the
    // four waves, then write this block's (max, sum) per row.
#pragma unroll
    for (int qt = 0; qt < kNqtMax; ++qt) {
      if (qt >= nqt) break;
      float m0 = mrun[qt], s0 = srun[qt];
#pragma unroll
      for (int msk = 16; msk <= 32; msk <<= 1) {
        float mo = __shfl_xor(m0, msk, 64);
        float so = __shfl_xor(s0, msk, 64);
        float mn = fmaxf(m0, mo);
        float sn = 0.f;
        if (mn != -INFINITY)
          sn = s0 * __builtin_amdgcn_exp2f(m0 - mn) + so * __builtin_amdgcn_exp2f(mo - mn);
        m0 = mn;
        s0 = sn;
      }
      if (grp == 0) {
        red_lds[(wave * Mp + qt * 16 + c16) * 2] = m0;
        red_lds[(wave * Mp + qt * 16 + c16) * 2 + 1] = s0;
      }
    }
    __syncthreads();
    for (int rho = threadIdx.x; rho < M; rho += kScoreThreads) {
      float mt = -INFINITY;
      for (int wv = 0; wv < 4; ++wv) mt = fmaxf(mt, red_lds[(wv * Mp + rho) * 2]);
      float sacc = 0.f;
      if (mt != -INFINITY) {
        for (int wv = 0; wv < 4; ++wv) {
          float mw = red_lds[(wv * Mp + rho) * 2];
          if (mw != -INFINITY) sacc += red_lds[(wv * Mp + rho) * 2 + 1] * __builtin_amdgcn_exp2f(mw - mt);
        }
      }
      part[(u * nkb_max + kb) * M + rho] = make_float2(mt, sacc);
    }
  } else if (kpart) {
    // Reduce the weighted key sums over the 16 lanes of each group, then over
    // the four waves.
    float v[QD];
#pragma unroll
    for (int i = 0; i < QD; ++i) v[i] = kacc[i];
#pragma unroll
    for (int m = 8, half = QD / 2; m >= 1; m >>= 1, half >>= 1) {
      const bool up = (lane & m) != 0;
#pragma unroll
      for (int i = 0; i < half; ++i) {
        float keep = up ? v[half + i] : v[i];
        float send = up ? v[i] : v[half + i];
        v[i] = keep + __shfl_xor(send, m, 64);
      }
    }
    constexpr int PER = QD / 16;  // dims left per lane
    __syncthreads();
#pragma unroll
    for (int e = 0; e < PER; ++e) red_lds[wave * D + grp * QD + c16 * PER + e] = v[e];
    __syncthreads();
    for (int dd = threadIdx.x; dd < D; dd += kScoreThreads) {
      float s = red_lds[dd] + red_lds[D + dd] + red_lds[2 * D + dd] + red_lds[3 * D + dd];
      kpart[(u * nkb_max + kb) * D + dd] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// Combine per-block (max, sum) into the per-row log2-sum-exp.
__global__ __launch_bounds__(256) void lse_combine_kernel(Geo g, SeqTab st, int32_t keys_per_block,
                                                           int32_t nkb_max,
                                                           const float2* __restrict__ part,
                                                           float* __restrict__ lse2) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int nkb = (n + keys_per_block - 1) / keys_per_block;
  const int M = g.w * g.G;
  const int64_t u = unit_index(g, l, b, h);
  for (int rho = threadIdx.x; rho < M; rho += blockDim.x) {
    float mt = -INFINITY;
    for (int kb = 0; kb < nkb; ++kb) mt = fmaxf(mt, part[(u * nkb_max + kb) * M + rho].x);
    float s = 0.f;
    for (int kb = 0; kb < nkb; ++kb) {
      float2 p = part[(u * nkb_max + kb) * M + rho];
      if (p.x != -INFINITY) s += p.y * __builtin_amdgcn_exp2f(p.x - mt);
    }
    lse2[u * M + rho] = mt + __builtin_amdgcn_logf(s);
  }
}

// Sum the per-block weighted key sums in fp64 (fixed block order).
__global__ __launch_bounds__(128) void ksum_reduce_kernel(Geo g, SeqTab st, int32_t keys_per_block,
                                                           int32_t nkb_max,
                                                           const float* __restrict__ kpart,
                                                           double* __restrict__ ksum) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int nkb = (n + keys_per_block - 1) / keys_per_block;
  const int64_t u = unit_index(g, l, b, h);
  for (int dd = threadIdx.x; dd < g.D; dd += blockDim.x) {
    double s = 0.0;
    for (int kb = 0; kb < nkb; ++kb) s += (double)kpart[(u * nkb_max + kb) * g.D + dd];
    ksum[u * g.D + dd] = s;
  }
}

// ---------------------------------------------------------------------------
// fp32 inputs: one key per thread, window queries in LDS, VALU dot products.
template <int D, bool P2>
__global__ __launch_bounds__(256) void score_f32_kernel(
    Geo g, SeqTab st, const float* __restrict__ qw, int64_t q_sl, int64_t q_st, int64_t q_sh,
    const float* __restrict__ kc, int64_t k_sl, int64_t k_st, int64_t k_sh, int32_t nkb_max,
    float2* __restrict__ part, const float* __restrict__ lse2, float* __restrict__ scores,
    float* __restrict__ kpart) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* q_lds = reinterpret_cast<float*>(smem_raw);
  const int kb = blockIdx.x;
  const int h = blockIdx.y % g.H;
  const int bl = blockIdx.y / g.H;
  const int l = blockIdx.z;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t tok0 = st.start[bl];
  if (kb * 256 >= n) return;
  const int M = g.w * g.G;
  const int64_t u = unit_index(g, l, b, h);
  float* lse_lds = q_lds + M * D;
  float* red = lse_lds + M;  // [8] + [4][D]
  for (int c = threadIdx.x; c < M * D; c += 256) {
    int rho = c / D, dd = c % D;
    int qq = rho / g.G, gq = rho % g.G;
    q_lds[c] = qw[(int64_t)l * q_sl + (int64_t)(b * g.w + qq) * q_st + (int64_t)(h * g.G + gq) * q_sh + dd];
  }
  if (P2)
    for (int i = threadIdx.x; i < M; i += 256) lse_lds[i] = lse2[u * M + i];
  __syncthreads();
  const int key = kb * 256 + threadIdx.x;
  const bool valid = key < n;
  const int keyc = valid ? key : n - 1;
  const float* krow = kc + (int64_t)l * k_sl + (tok0 + keyc) * k_st + (int64_t)h * k_sh;
  float kr[D];
#pragma unroll
  for (int t = 0; t < D; ++t) kr[t] = krow[t];
  const float c2 = g.scale * kLog2e;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float s_acc = 0.f;
  for (int rho = 0; rho < M; ++rho) {
    const float* qr = q_lds + rho * D;
    float dot = 0.f;
#pragma unroll
    for (int t = 0; t < D; ++t) dot = fmaf(qr[t], kr[t], dot);
    const int qpos = n - g.w + rho / g.G;
    const bool vis = valid && (!g.causal || key <= qpos);
    const float x = dot * c2;
    if (!P2) {
      float mx = wave_max(vis ? x : -INFINITY);
      if (lane == 0) red[wave] = mx;
      __syncthreads();
      float mt = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      __syncthreads();
      float e = (vis && mt != -INFINITY) ? __builtin_amdgcn_exp2f(x - mt) : 0.f;
      float sw = wave_sum(e);
      if (lane == 0) red[wave] = sw;
      __syncthreads();
      if (threadIdx.x == 0)
        part[(u * nkb_max + kb) * M + rho] = make_float2(mt, red[0] + red[1] + red[2] + red[3]);
      __syncthreads();
    } else {
      if (vis) s_acc += __builtin_amdgcn_exp2f(x - lse_lds[rho]);
    }
  }
  if (P2) {
    if (valid) scores[lht_base(g, l, h, tok0) + key] = s_acc;
    if (kpart) {
      const float sp = (valid && s_acc > 0.f) ? s_acc : 0.f;
      float* wred = red + 8;
#pragma unroll
      for (int t = 0; t < D; ++t) {
        float x = wave_sum(sp * kr[t]);
        if (lane == 0) wred[wave * D + t] = x;
      }
      __syncthreads();
      for (int t = threadIdx.x; t < D; t += 256)
        kpart[(u * nkb_max + kb) * D + t] = wred[t] + wred[D + t] + wred[2 * D + t] + wred[3 * D + t];
    }
  }
}

// ---------------------------------------------------------------------------
// Host side.


size_t score_smem_bytes(const Geo& g, int32_t dtype) {
  const int M = g.w * g.G;
  if (dtype == CERTKV_BF16) {
    const size_t Mp = (size_t)((M + 15) & ~15);
    size_t q = Mp * (g.D + 8) * 2;
    size_t red = (size_t)4 * (Mp * 2 > (size_t)g.D ? Mp * 2 : (size_t)g.D) * 4;
    return q + Mp * 4 + red;
  }
  return (size_t)M * g.D * 4 + (size_t)M * 4 + 8 * 4 + (size_t)4 * g.D * 4;
}

template <int D>
static certkv_status launch_mfma(const ScoreArgs& a, const SeqTab& st, int max_len,
                                 hipStream_t s) {
  const Geo& g = a.g;
  const int nkb = (max_len + a.keys_per_block - 1) / a.keys_per_block;
  dim3 grid(nkb, g.H * st.count, g.L);
  size_t smem = score_smem_bytes(g, CERTKV_BF16);
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncSetAttribute((const void*)score_mfma_kernel<D, false>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    hipFuncSetAttribute((const void*)score_mfma_kernel<D, true>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    attr_set = true;
  }
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* k = static_cast<const uint16_t*>(a.k.ptr);
  CERTKV_LAUNCH("score_pass1_mfma", (score_mfma_kernel<D, false>), grid, dim3(kScoreThreads), smem,
                s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token,
                a.k.s_head, a.keys_per_block, a.nkb_max, a.part, (const float*)nullptr,
                (float*)nullptr, (float*)nullptr);
  CERTKV_LAUNCH("score_lse_combine", lse_combine_kernel, dim3(g.H * st.count, g.L), dim3(256), 0, s,
                g, st, a.keys_per_block, a.nkb_max, (const float2*)a.part, a.lse2);
  CERTKV_LAUNCH("score_pass2_mfma", (score_mfma_kernel<D, true>), grid, dim3(kScoreThreads), smem,
                s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token,
                a.k.s_head, a.keys_per_block, a.nkb_max, (float2*)nullptr, (const float*)a.lse2,
                a.scores, a.ksum ? a.kpart : (float*)nullptr);
  if (a.ksum)
    CERTKV_LAUNCH("score_ksum_reduce", ksum_reduce_kernel, dim3(g.H * st.count, g.L), dim3(128), 0,
                  s, g, st, a.keys_per_block, a.nkb_max, (const float*)a.kpart, a.ksum);
  return CERTKV_OK;
}

template <int D>
static certkv_status launch_f32(const ScoreArgs& a, const SeqTab& st, int max_len, hipStream_t s) {
  const Geo& g = a.g;
  const int nkb = (max_len + 255) / 256;
  dim3 grid(nkb, g.H * st.count, g.L);
  size_t smem = score_smem_bytes(g, CERTKV_F32);
  const float* q = static_cast<const float*>(a.q.ptr);
  const float* k = static_cast<const float*>(a.k.ptr);
  CERTKV_LAUNCH("score_pass1_f32", (score_f32_kernel<D, false>), grid, dim3(256), smem, s, g, st, q,
                a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token, a.k.s_head,
                a.nkb_max, a.part, (const float*)nullptr, (float*)nullptr, (float*)nullptr);
  CERTKV_LAUNCH("score_lse_combine", lse_combine_kernel, dim3(g.H * st.count, g.L), dim3(256), 0, s,
                g, st, 256, a.nkb_max, (const float2*)a.part, a.lse2);
  CERTKV_LAUNCH("score_pass2_f32", (score_f32_kernel<D, true>), grid, dim3(256), smem, s, g, st, q,
                a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token, a.k.s_head,
                a.nkb_max, (float2*)nullptr, (const float*)a.lse2, a.scores,
                a.ksum ? a.kpart : (float*)nullptr);
  if (a.ksum)
    CERTKV_LAUNCH("score_ksum_reduce", ksum_reduce_kernel, dim3(g.H * st.count, g.L), dim3(128), 0,
                  s, g, st, 256, a.nkb_max, (const float*)a.kpart, a.ksum);
  return CERTKV_OK;
}

certkv_status run_score(const ScoreArgs& a, const SeqTab& st, int max_len, hipStream_t s) {
  if (a.dtype == CERTKV_F32)
    return a.g.D == 128 ? launch_f32<128>(a, st, max_len, s) : launch_f32<64>(a, st, max_len, s);
  if (a.g.D == 128) return launch_mfma<128>(a, st, max_len, s);
  return launch_mfma<64>(a, st, max_len, s);
}

}  // namespace certkv
