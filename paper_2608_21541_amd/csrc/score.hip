// Observation-window scoring on gfx950.
//
// For KV head h the M = w*G window rows (query head g of the group, window
// position q) give logits l = scale * <q_row, k_j>; the score of key j is the
// sum over rows of the row-softmax weight of key j.  Two passes over K:
//   pass 1   per key block: sum over the block of exp2(l * log2 e) per row;
//   combine  per row: log2 of the sum over blocks;
//   pass 2   per key block: s_j = sum_rows exp2(l_row,j * log2 e - lse2_row),
//            written out, plus (optionally) the block's sum_j s_j k_j.
// Pass 1 sums exponentials without a running maximum, so partial sums of
// different blocks add directly.  A row whose total falls outside
// [2^-60, 2^120] (where fp32 exponentials could under- or overflow) flags its
// unit, and a fallback pass recomputes that unit's partials with a running
// maximum; it returns immediately for units that are not flagged.
// The contraction runs on MFMA v_mfma_f32_32x32x16_bf16 with the key tile in
// VGPRs straight from HBM and the window queries staged once per workgroup in
// LDS.  Pass 1 makes the key tile the A operand, so each lane owns one query
// column and row sums are lane-local; pass 2 makes it the B operand, so each
// lane owns one key and per-key sums are lane-local.
#include <type_traits>

#include "stages.h"

namespace certkv {

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16_t __attribute__((__vector_size__(16 * sizeof(float))));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kScoreThreads = 512;  // 8 waves
constexpr float kSumLo = 8.673617379884035e-19f;  // 2^-60
constexpr float kSumHi = 1.329227995784916e+36f;  // 2^120

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

enum { kPass1Sum = 0, kPass1Max = 1 };

// One round of a transpose-reduce over lane bit M: lanes with that bit set
// keep the upper HALF of their 2*HALF values, the others the lower HALF, and
// each adds its partner's copy of the half it keeps.  The rounds recurse at
// compile time (HALF and M halve) so that every register index is a constant.
template <int HALF, int M>
__device__ __forceinline__ void xpose_round(float* v, int lane) {
  const bool up = (lane & M) != 0;
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const float keep = up ? v[HALF + i] : v[i];
    const float send = up ? v[i] : v[HALF + i];
    v[i] = keep + __shfl_xor(send, M, 64);
  }
  if constexpr (HALF > 1 && M > 1) xpose_round<HALF / 2, M / 2>(v, lane);
}

// MFMA v_mfma_f32_32x32x16_bf16 layout used below (per 64-lane wave):
//   A (32 keys x 16 dims): lane (hh = lane/32, c = lane%32) supplies key c,
//     8 dims of its half's slice;
//   B (16 dims x 32 queries): the same lane supplies query c, same dims;
//   D (32 x 32): lane (hh, c) holds query column c, key rows
//     8*(v/4) + 4*hh + v%4 for v = 0..15.
// The contraction order is free, so lane half hh owns the contiguous dims
// hh*D/2 .. hh*D/2 + D/2 - 1 for all of its k-steps: a lane loads one D-byte
// run of its key row, and k-step s takes its dims 8*s .. 8*s + 7.
template <int D, int NQT, int MODE>
__global__ __launch_bounds__(kScoreThreads) __attribute__((amdgpu_waves_per_eu(NQT > 8 ? 2 : 4, 8))) void score_mfma_kernel(
    Geo g, SeqTab st, const uint16_t* __restrict__ qw, int64_t q_sl, int64_t q_st,
    int64_t q_sh, const uint16_t* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, int32_t keys_per_block, int32_t nkb_max, float2* __restrict__ part,
    const int32_t* __restrict__ flag) {
  constexpr int KS = D / 16;   // MFMA k-steps
  constexpr int HD = D / 2;    // dims per lane half
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
  const int Mp = NQT * 32;  // rows padded to whole 32-query tiles
  const int64_t u = unit_index(g, l, b, h);
  if (MODE == kPass1Max && flag[u] == 0) return;

  int* lim_lds = reinterpret_cast<int*>(smem_raw + (size_t)Mp * RE * 2 + (size_t)Mp * 4);
  // Cross-wave reduction area, aliasing the staged queries once the key loop
  // is done: [8][Mp] sums or [8][Mp][2] (max, sum) pairs.
  float* red_lds = reinterpret_cast<float*>(smem_raw);

  // Stage the window queries of this KV head: row rho = q*G + gq; padding
  // rows are zero and are never written out.
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
    // Last visible key of each row: the causal limit of its window position,
    // -1 for padding rows.
    for (int i = threadIdx.x; i < Mp; i += kScoreThreads) {
      int lim = -1;
      if (i < M) lim = g.causal ? min(n - g.w + i / g.G, n - 1) : n - 1;
      lim_lds[i] = lim;
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  const float c2 = g.scale * kLog2e;
  const int first_masked = g.causal ? (n - g.w + 1) : n;  // keys >= this may be masked
  const uint16_t* kbase = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;

  float srun[NQT];  // this lane's query column, per query tile
  float mrun[MODE == kPass1Max ? NQT : 1];
#pragma unroll
  for (int i = 0; i < NQT; ++i) srun[i] = 0.f;
#pragma unroll
  for (int i = 0; i < (MODE == kPass1Max ? NQT : 1); ++i) mrun[i] = -INFINITY;

  constexpr int KPW = 32;             // keys per wave iteration
  constexpr int KPI = KPW * kScoreThreads / 64;  // keys per workgroup iteration
  for (int it = key_begin + wave * KPW; it < key_end; it += KPI) {
    // The 32-key tile (keys it..it+31) as A fragments, straight from HBM.
    Frag kf[KS];
    {
      const int key = it + c32;
      const int keyc = key < n ? key : n - 1;
      const uint4* src = reinterpret_cast<const uint4*>(kbase + (int64_t)keyc * k_st + hh * HD);
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[s].u = src[s];
    }
    const bool need_mask = (it + KPW - 1 >= first_masked) || (it + KPW - 1 >= n);

    // The query-tile loop is software-pipelined: the MFMA chain of tile qt+1
    // is interleaved with the masking and exponentials of tile qt (a slice
    // of 16/KS values behind each MFMA), so that the matrix core and the VALU
    // of one wave work at once; gfx950 overlaps them within a wave, not
    // across waves.  It is instantiated with and without the causal / tail
    // mask so that no branch splits it.
    auto tiles = [&](auto masked_tag) {
      constexpr bool MASKED = decltype(masked_tag)::value;
      constexpr int SL = 16 / KS;  // values of the current tile per k-step
      // value v of the current tile's accumulator, masked and scaled
      auto logit = [&](const f32x16_t& acc, int v, int lim) {
        float x = acc[v];
        if (MASKED && it + 8 * (v >> 2) + 4 * hh + (v & 3) > lim) x = -INFINITY;
        return x;
      };
      f32x16_t acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.f;
      {
        const uint16_t* qrow = q_lds + c32 * RE + hh * HD;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          Frag qf;
          qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf.v, acc, 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        const bool more = qt + 1 < NQT;
        const int lim = MASKED ? lim_lds[qt * 32 + c32] : 0;
        f32x16_t nacc;
#pragma unroll
        for (int v = 0; v < 16; ++v) nacc[v] = 0.f;
        const uint16_t* qrow = q_lds + ((qt + 1) * 32 + c32) * RE + hh * HD;
        if (MODE == kPass1Max) {
          // fallback pass: a running maximum needs the whole tile first
          if (more) {
#pragma unroll
            for (int s = 0; s < KS; ++s) {
              Frag qf;
              qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
              nacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf.v, nacc, 0, 0, 0);
            }
          }
          float mx = logit(acc, 0, lim);
#pragma unroll
          for (int v = 1; v < 16; ++v) mx = fmaxf(mx, logit(acc, v, lim));
          const float mnew = fmaxf(mrun[qt], mx * c2);
          if (mnew != -INFINITY) {
            const float sc = __builtin_amdgcn_exp2f(mrun[qt] - mnew);
            float sacc = 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v)
              sacc += __builtin_amdgcn_exp2f(fmaf(logit(acc, v, lim), c2, -mnew));
            srun[qt] = fmaf(srun[qt], sc, sacc);
            mrun[qt] = mnew;
          }
        } else {
          float sacc = 0.f;
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            if (more) {
              Frag qf;
              qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
              nacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf.v, nacc, 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < SL; ++j) {
              const int v = s * SL + j;
              sacc += __builtin_amdgcn_exp2f(logit(acc, v, lim) * c2);
            }
          }
          srun[qt] += sacc;
          if (more) {
            // LDS reads two k-steps ahead of their MFMA, each k-step's VALU
            // slice right behind its MFMA.
            __builtin_amdgcn_sched_group_barrier(0x100, 2 + (MASKED ? 1 : 0), 0);
#pragma unroll
            for (int s = 0; s < KS; ++s) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x402, (MASKED ? 5 : 3) * SL, 0);
              if (s + 2 < KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
          }
        }
        acc = nacc;
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if (need_mask)
      tiles(std::integral_constant<bool, true>());
    else
      tiles(std::integral_constant<bool, false>());
  }

  constexpr int NW = kScoreThreads / 64;
  __syncthreads();  // every wave is done with the staged queries
  if (MODE == kPass1Sum) {
    // Sum the two lane halves (same query column), then the waves.
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      float s0 = srun[qt];
      s0 += __shfl_xor(s0, 32, 64);
      if (hh == 0) red_lds[wave * Mp + qt * 32 + c32] = s0;
    }
    __syncthreads();
    for (int rho = threadIdx.x; rho < M; rho += kScoreThreads) {
      float sacc = 0.f;
      for (int wv = 0; wv < NW; ++wv) sacc += red_lds[wv * Mp + rho];
      part[(u * nkb_max + kb) * M + rho] = make_float2(sacc, 0.f);
    }
  } else if (MODE == kPass1Max) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      float m0 = mrun[qt], s0 = srun[qt];
      const float mo = __shfl_xor(m0, 32, 64);
      const float so = __shfl_xor(s0, 32, 64);
      const float mn = fmaxf(m0, mo);
      float sn = 0.f;
      if (mn != -INFINITY)
        sn = s0 * __builtin_amdgcn_exp2f(m0 - mn) + so * __builtin_amdgcn_exp2f(mo - mn);
      if (hh == 0) {
        red_lds[(wave * Mp + qt * 32 + c32) * 2] = mn;
        red_lds[(wave * Mp + qt * 32 + c32) * 2 + 1] = sn;
      }
    }
    __syncthreads();
    for (int rho = threadIdx.x; rho < M; rho += kScoreThreads) {
      float mt = -INFINITY;
      for (int wv = 0; wv < NW; ++wv) mt = fmaxf(mt, red_lds[(wv * Mp + rho) * 2]);
      float sacc = 0.f;
      if (mt != -INFINITY) {
        for (int wv = 0; wv < NW; ++wv) {
          float mw = red_lds[(wv * Mp + rho) * 2];
          if (mw != -INFINITY) sacc += red_lds[(wv * Mp + rho) * 2 + 1] * __builtin_amdgcn_exp2f(mw - mt);
        }
      }
      part[(u * nkb_max + kb) * M + rho] = make_float2(mt, sacc);
    }
  }
}

// ---------------------------------------------------------------------------
// Pass 2 with the operands swapped: the window queries are the A operand
// (rows = 32 queries of a tile, from LDS) and the key tile the B operand
// (columns = 32 keys, in VGPRs straight from HBM).  Lane (hh, c) then holds
// key c of the tile and the query rows 8*(v/4) + 4*hh + v%4 (v = 0..15) of
// every query tile, so a key's score is a lane-local sum over its rows plus
// one exchange between the two lane halves, and its weighted key row is
// already in the lane's registers.  With the key sums (64 accumulators per
// lane) the kernel runs two waves per SIMD and loads the next key tile while
// the current one is consumed; without them (and for windows of at most 256
// rows) it keeps four waves per SIMD and lets the other waves hide the load
// latency.
template <int D, int NQT, bool KSUM>
__global__ __launch_bounds__(kScoreThreads) __attribute__((amdgpu_waves_per_eu((KSUM || NQT > 8) ? 2 : 4, 8))) void score_pass2_kernel(
    Geo g, SeqTab st, const uint16_t* __restrict__ qw, int64_t q_sl, int64_t q_st,
    int64_t q_sh, const uint16_t* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, int32_t keys_per_block, int32_t nkb_max, const float* __restrict__ lse2,
    float* __restrict__ scores, float* __restrict__ kpart) {
  constexpr int KS = D / 16;   // MFMA k-steps
  constexpr int HD = D / 2;    // dims per lane half
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
  const int Mp = NQT * 32;
  const int64_t u = unit_index(g, l, b, h);

  float* lse_lds = reinterpret_cast<float*>(smem_raw + (size_t)Mp * RE * 2);
  int* lim_lds = reinterpret_cast<int*>(lse_lds + Mp);
  float* red_lds = reinterpret_cast<float*>(smem_raw);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  const uint16_t* kbase = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;
  constexpr int KPW = 32;                        // keys per wave iteration
  constexpr int KPI = KPW * kScoreThreads / 64;  // keys per workgroup iteration
  // Key tile starting at `it` (rows clamped into the sequence) into kf.
  auto load_tile = [&](int it, Frag(&kf)[KS]) {
    const int key = it + c32;
    const int keyc = key < n ? key : n - 1;
    const uint4* src = reinterpret_cast<const uint4*>(kbase + (int64_t)keyc * k_st + hh * HD);
#pragma unroll
    for (int s = 0; s < KS; ++s) kf[s].u = src[s];
  };
  Frag kf[KS], kn[KSUM ? KS : 1];
  const int it0 = key_begin + wave * KPW;
  if (it0 < key_end) load_tile(it0, kf);

  // Stage the window queries (row rho = q*G + gq, zero padding rows), the
  // row log2-sums (+inf for padding rows, whose weights are then zero) and
  // the causal limits.
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
    for (int i = threadIdx.x; i < Mp; i += kScoreThreads) {
      int lim = -1;
      if (i < M) lim = g.causal ? min(n - g.w + i / g.G, n - 1) : n - 1;
      lim_lds[i] = lim;
      lse_lds[i] = i < M ? lse2[u * M + i] : INFINITY;
    }
  }
  __syncthreads();

  const float c2 = g.scale * kLog2e;
  const int first_masked = g.causal ? (n - g.w + 1) : n;  // keys >= this may be masked
  float kacc[KSUM ? HD : 1];
#pragma unroll
  for (int i = 0; i < (KSUM ? HD : 1); ++i) kacc[i] = 0.f;

  for (int it = it0; it < key_end; it += KPI) {
    if constexpr (KSUM) {
      if (it + KPI < key_end) load_tile(it + KPI, kn);
    } else {
      if (it != it0) load_tile(it, kf);
    }
    const bool need_mask = it + KPW - 1 >= first_masked;
    float sp[16 / KS];  // this lane's key: sums over its rows (independent chains)
#pragma unroll
    for (int j = 0; j < 16 / KS; ++j) sp[j] = 0.f;

    // Query tiles software-pipelined as in pass 1: the MFMA chain of tile
    // qt+1 interleaved with the exponentials of tile qt.
    auto tiles = [&](auto masked_tag) {
      constexpr bool MASKED = decltype(masked_tag)::value;
      constexpr int SL = 16 / KS;  // values of the current tile per k-step
      const int key = it + c32;
      f32x16_t acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.f;
      {
        const uint16_t* qrow = q_lds + c32 * RE + hh * HD;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          Frag qf;
          qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.v, kf[s].v, acc, 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        const bool more = qt + 1 < NQT;
        // rows of value v: qt*32 + 4*hh + 8*(v/4) + v%4, four runs of four
        const int rb = qt * 32 + 4 * hh;
        float4 l2[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) l2[i] = *reinterpret_cast<const float4*>(lse_lds + rb + 8 * i);
        int4 lim[4];
        if (MASKED) {
#pragma unroll
          for (int i = 0; i < 4; ++i) lim[i] = *reinterpret_cast<const int4*>(lim_lds + rb + 8 * i);
        }
        f32x16_t nacc;
#pragma unroll
        for (int v = 0; v < 16; ++v) nacc[v] = 0.f;
        const uint16_t* qrow = q_lds + ((qt + 1) * 32 + c32) * RE + hh * HD;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          if (more) {
            Frag qf;
            qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
            nacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.v, kf[s].v, nacc, 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < SL; ++j) {
            const int v = s * SL + j;
            const float4 lv = l2[v >> 2];
            const float lsev = (v & 3) == 0 ? lv.x : (v & 3) == 1 ? lv.y : (v & 3) == 2 ? lv.z : lv.w;
            float x = acc[v];
            if (MASKED) {
              const int4 mv = lim[v >> 2];
              const int limv = (v & 3) == 0 ? mv.x : (v & 3) == 1 ? mv.y : (v & 3) == 2 ? mv.z : mv.w;
              if (key > limv) x = -INFINITY;
            }
            sp[j] += __builtin_amdgcn_exp2f(fmaf(x, c2, -lsev));
          }
        }
        if (more) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2 + 4 + (MASKED ? 4 : 0), 0);
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x402, (MASKED ? 5 : 3) * SL, 0);
            if (s + 2 < KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
        }
        acc = nacc;
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if (need_mask)
      tiles(std::integral_constant<bool, true>());
    else
      tiles(std::integral_constant<bool, false>());

    float sp_all = sp[0];
#pragma unroll
    for (int j = 1; j < 16 / KS; ++j) sp_all += sp[j];
    const float s_key = sp_all + __shfl_xor(sp_all, 32, 64);
    const int key = it + c32;
    if (hh == 0 && key < n) scores[lht_base(g, l, h, tok0) + key] = s_key;
    if constexpr (KSUM) {
      const float s_t = (key < n && s_key > 0.f) ? s_key : 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint32_t* w4 = reinterpret_cast<const uint32_t*>(&kf[s].u);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kacc[s * 8 + 2 * e] = fmaf(s_t, bf16_lo(w4[e]), kacc[s * 8 + 2 * e]);
          kacc[s * 8 + 2 * e + 1] = fmaf(s_t, bf16_hi(w4[e]), kacc[s * 8 + 2 * e + 1]);
        }
      }
    }
    if constexpr (KSUM) {
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[s].u = kn[s].u;
    }
  }

  if constexpr (KSUM) {
    constexpr int NW = kScoreThreads / 64;
    __syncthreads();  // every wave is done with the staged queries
    // Sum the weighted key rows over the 32 keys of each lane half (a
    // transpose-reduce leaves dims hh*HD + c32*PER + e in lane (hh, c32)),
    // then over the waves.
    float v[HD];
#pragma unroll
    for (int i = 0; i < HD; ++i) v[i] = kacc[i];
    xpose_round<HD / 2, 16>(v, lane);
    constexpr int PER = HD / 32;
#pragma unroll
    for (int e = 0; e < PER; ++e) red_lds[wave * D + hh * HD + c32 * PER + e] = v[e];
    __syncthreads();
    for (int dd = threadIdx.x; dd < D; dd += kScoreThreads) {
      float s = 0.f;
      for (int wv = 0; wv < NW; ++wv) s += red_lds[wv * D + dd];
      kpart[(u * nkb_max + kb) * D + dd] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// Pass 2 for windows of at most 256 rows: sixteen waves per workgroup (four
// per SIMD at one workgroup per CU) share one copy of the staged queries.
// The layout is score_pass2_kernel's (query tile = A, key tile = B, one key
// per lane), with two changes that free the registers a fourth wave needs:
//  * the row log2-sums enter as the accumulators' starting value, -lse2 / c2,
//    so the exponent of a weight is one multiply of the MFMA result;
//  * the weighted key sums run on the matrix core.  After a tile's scores are
//    known, each wave stages its key tile in LDS 64 dims at a time and adds
//    s^T K with v_mfma_f32_4x4x4bf16_1k: block b of the instruction covers
//    dims 4b..4b+3 of the stage and 4 keys, the rows of A are the scores
//    split into three bf16 parts (hi + lo + lo2 = s exactly) and a zero row,
//    and the B fragments (4 keys x 4 dims per block) come from transposing
//    LDS reads (ds_read_b64_tr_b16: in each 16-lane group, lane i receives
//    element i % 4 of the 8-byte rows addressed by lanes 4j + i / 4).
// Per lane the key sums then take two 4-register accumulators instead of
// half a key row of fp32 sums.
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kP2Threads = 1024;
constexpr int kP2Waves = kP2Threads / 64;
constexpr int kStageRow = 160;  // bytes per staged key row: 64 dims + 32 B (an 8-bank shift)

template <int D, int NQT>
struct P2Smem {
  static constexpr int Mp = NQT * 32;
  static constexpr size_t lse = (size_t)Mp * ScoreSmem<D>::kRowElems * 2;  // [Mp] -lse2 / c2
  static constexpr size_t lim = lse + (size_t)Mp * 4;                      // [Mp] causal limits
  static constexpr size_t stage = lim + (size_t)Mp * 4;                    // [waves][32 keys][kStageRow]
  static constexpr size_t sparts = stage + (size_t)kP2Waves * 32 * kStageRow;  // [waves][4][32] bf16
  static constexpr size_t total = sparts + (size_t)kP2Waves * 4 * 32 * 2;
};

__device__ __forceinline__ s16x4_t lds_tr_b16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4_t*)(__attribute__((address_space(3))) unsigned char*)p);
}

template <int D, int NQT, bool KSUM>
__global__ __launch_bounds__(kP2Threads) __attribute__((amdgpu_waves_per_eu(4, 8))) void score_pass2_w16_kernel(
    Geo g, SeqTab st, const uint16_t* __restrict__ qw, int64_t q_sl, int64_t q_st,
    int64_t q_sh, const uint16_t* __restrict__ kc, int64_t k_sl, int64_t k_st,
    int64_t k_sh, int32_t keys_per_block, int32_t nkb_max, const float* __restrict__ lse2,
    float* __restrict__ scores, float* __restrict__ kpart) {
  using SM = P2Smem<D, NQT>;
  constexpr int KS = D / 16;   // MFMA k-steps
  constexpr int HD = D / 2;    // dims per lane half
  constexpr int RE = ScoreSmem<D>::kRowElems;
  constexpr int NSTG = D / 64; // key-sum stages of 64 dims
  static_assert(NQT <= 8, "sixteen-wave pass 2 holds at most 256 window rows");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  uint16_t* q_lds = reinterpret_cast<uint16_t*>(smem_raw);
  float* nl_lds = reinterpret_cast<float*>(smem_raw + SM::lse);
  int* lim_lds = reinterpret_cast<int*>(smem_raw + SM::lim);
  float* red_lds = reinterpret_cast<float*>(smem_raw);

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
  const int Mp = NQT * 32;
  const int64_t u = unit_index(g, l, b, h);
  const float c2 = g.scale * kLog2e;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  unsigned char* stage = smem_raw + SM::stage + (size_t)wave * 32 * kStageRow;
  uint16_t* sparts = reinterpret_cast<uint16_t*>(smem_raw + SM::sparts) + wave * 4 * 32;

  // Stage the window queries (row rho = q*G + gq, zero padding rows), the
  // accumulator starting values -lse2 / c2 (-infinity for padding rows,
  // whose weights are then zero) and the causal limits; zero the fourth row
  // of every wave's score parts.
  {
    const int chunks = D / 8;
    for (int c = threadIdx.x; c < Mp * chunks; c += kP2Threads) {
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
    for (int i = threadIdx.x; i < Mp; i += kP2Threads) {
      int lim = -1;
      if (i < M) lim = g.causal ? min(n - g.w + i / g.G, n - 1) : n - 1;
      lim_lds[i] = lim;
      nl_lds[i] = i < M ? -lse2[u * M + i] / c2 : -INFINITY;
    }
    if (KSUM && lane < 32) sparts[3 * 32 + lane] = 0;
  }
  __syncthreads();

  const int first_masked = g.causal ? (n - g.w + 1) : n;  // keys >= this may be masked
  const uint16_t* kbase = kc + (int64_t)l * k_sl + tok0 * k_st + (int64_t)h * k_sh;
  constexpr int KPW = 32;                    // keys per wave iteration
  constexpr int KPI = KPW * kP2Waves;        // keys per workgroup iteration
  f32x4_t kacc[NSTG];
#pragma unroll
  for (int i = 0; i < NSTG; ++i) kacc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // transposing-read address of this lane in a stage: key row 4t + (lane % 16) / 4,
  // 8-byte column chunk 4 (lane / 16) + lane % 4
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 8 * (4 * (lane >> 4) + (lane & 3));

  for (int it = key_begin + wave * KPW; it < key_end; it += KPI) {
    Frag kf[KS];
    {
      const int key = it + c32;
      const int keyc = key < n ? key : n - 1;
      const uint4* src = reinterpret_cast<const uint4*>(kbase + (int64_t)keyc * k_st + hh * HD);
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[s].u = src[s];
    }
    const bool need_mask = it + KPW - 1 >= first_masked;
    float sp[16 / KS];
#pragma unroll
    for (int j = 0; j < 16 / KS; ++j) sp[j] = 0.f;

    auto tiles = [&](auto masked_tag) {
      constexpr bool MASKED = decltype(masked_tag)::value;
      constexpr int SL = 16 / KS;
      const int key = it + c32;
      // accumulator starting values of query tile qt: rows qt*32 + 4*hh +
      // 8*(v/4) + v%4 of -lse2 / c2
      auto init_acc = [&](int qt, f32x16_t& a) {
        const int rb = qt * 32 + 4 * hh;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float4 x = *reinterpret_cast<const float4*>(nl_lds + rb + 8 * i);
          a[4 * i] = x.x;
          a[4 * i + 1] = x.y;
          a[4 * i + 2] = x.z;
          a[4 * i + 3] = x.w;
        }
      };
      f32x16_t acc;
      init_acc(0, acc);
      {
        const uint16_t* qrow = q_lds + c32 * RE + hh * HD;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          Frag qf;
          qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.v, kf[s].v, acc, 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        const bool more = qt + 1 < NQT;
        const int rb = qt * 32 + 4 * hh;
        int4 lim[4];
        if (MASKED) {
#pragma unroll
          for (int i = 0; i < 4; ++i) lim[i] = *reinterpret_cast<const int4*>(lim_lds + rb + 8 * i);
        }
        f32x16_t nacc;
        if (more) init_acc(qt + 1, nacc);
        const uint16_t* qrow = q_lds + ((qt + 1) * 32 + c32) * RE + hh * HD;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          if (more) {
            Frag qf;
            qf.u = *reinterpret_cast<const uint4*>(qrow + s * 8);
            nacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf.v, kf[s].v, nacc, 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < SL; ++j) {
            const int v = s * SL + j;
            float x = acc[v] * c2;
            if (MASKED) {
              const int4 mv = lim[v >> 2];
              const int limv = (v & 3) == 0 ? mv.x : (v & 3) == 1 ? mv.y : (v & 3) == 2 ? mv.z : mv.w;
              if (key > limv) x = -INFINITY;
            }
            sp[j] += __builtin_amdgcn_exp2f(x);
          }
        }
        if (more) {
          // every query fragment of the next tile read up front (measured
          // faster here than two steps ahead), then per k-step one MFMA and
          // the current tile's terms of that slice
          __builtin_amdgcn_sched_group_barrier(0x100, KS + 4 + (MASKED ? 4 : 0), 0);
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x402, (MASKED ? 5 : 3) * SL, 0);
          }
        }
        acc = nacc;
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if (need_mask)
      tiles(std::integral_constant<bool, true>());
    else
      tiles(std::integral_constant<bool, false>());

    float sp_all = sp[0];
#pragma unroll
    for (int j = 1; j < 16 / KS; ++j) sp_all += sp[j];
    const float s_key = sp_all + __shfl_xor(sp_all, 32, 64);
    const int key = it + c32;
    if (hh == 0 && key < n) scores[lht_base(g, l, h, tok0) + key] = s_key;
    if constexpr (KSUM) {
      // s = hi + lo + lo2 exactly (three bf16 parts of the fp32 value)
      const float s_t = (key < n && s_key > 0.f) ? s_key : 0.f;
      const uint16_t p0 = f32_to_bf16_rne(s_t);
      const float r1 = s_t - bf16_to_f32(p0);
      const uint16_t p1 = f32_to_bf16_rne(r1);
      const float r2 = r1 - bf16_to_f32(p1);
      const uint16_t p2 = f32_to_bf16_rne(r2);
      if (hh == 0) {
        sparts[c32] = p0;
        sparts[32 + c32] = p1;
        sparts[64 + c32] = p2;
      }
#pragma unroll
      for (int sg = 0; sg < NSTG; ++sg) {
        // stage 64 dims of the 32 keys: for d = 128 the lane half hh == sg
        // holds them (dims 64 sg ..), for d = 64 both halves write theirs
        if (NSTG == 1 || hh == sg) {
#pragma unroll
          for (int s = 0; s < KS; ++s)
            *reinterpret_cast<uint4*>(stage + c32 * kStageRow + (NSTG == 1 ? hh * 64 : 0) + 16 * s) =
                kf[s].u;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const s16x4_t a = *reinterpret_cast<const s16x4_t*>(sparts + (lane & 3) * 32 + 4 * t);
          const s16x4_t bfr = lds_tr_b16(stage + (4 * t + tr_row) * kStageRow + tr_col);
          kacc[sg] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a, bfr, kacc[sg], 0, 0, 0);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
  }

  if constexpr (KSUM) {
    __syncthreads();  // every wave is done with the staged queries
    // lane L holds dim 64 sg + L of stage sg: the sum of its three part rows
#pragma unroll
    for (int sg = 0; sg < NSTG; ++sg)
      red_lds[wave * D + 64 * sg + lane] = kacc[sg][0] + kacc[sg][1] + kacc[sg][2];
    __syncthreads();
    for (int dd = threadIdx.x; dd < D; dd += kP2Threads) {
      float s = 0.f;
      for (int wv = 0; wv < kP2Waves; ++wv) s += red_lds[wv * D + dd];
      kpart[(u * nkb_max + kb) * D + dd] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// Per-row log2-sum-exp from the pass-1 partials.
// Sum format (shift-free partial sums): writes lse2 and flags the unit when a
// row's total leaves [2^-60, 2^120].  Max format ((max, sum) partials):
// combines with rescaling; with `only_flagged` it touches flagged units only.
template <bool SUM_FORMAT>
__global__ __launch_bounds__(256) void lse_combine_kernel(Geo g, SeqTab st, int32_t keys_per_block,
                                                           int32_t nkb_max,
                                                           const float2* __restrict__ part,
                                                           float* __restrict__ lse2,
                                                           int32_t* __restrict__ flag,
                                                           int32_t only_flagged) {
  __shared__ int bad;
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int nkb = (n + keys_per_block - 1) / keys_per_block;
  const int M = g.w * g.G;
  const int64_t u = unit_index(g, l, b, h);
  if (!SUM_FORMAT && only_flagged && flag[u] == 0) return;
  if (SUM_FORMAT && threadIdx.x == 0) bad = 0;
  __syncthreads();
  for (int rho = threadIdx.x; rho < M; rho += blockDim.x) {
    if (SUM_FORMAT) {
      float s = 0.f;
      for (int kb = 0; kb < nkb; ++kb) s += part[(u * nkb_max + kb) * M + rho].x;
      if (!(s >= kSumLo && s <= kSumHi)) bad = 1;
      lse2[u * M + rho] = __builtin_amdgcn_logf(s);
    } else {
      float mt = -INFINITY;
      for (int kb = 0; kb < nkb; ++kb) mt = fmaxf(mt, part[(u * nkb_max + kb) * M + rho].x);
      float s = 0.f;
      for (int kb = 0; kb < nkb; ++kb) {
        float2 p = part[(u * nkb_max + kb) * M + rho];
        if (p.x != -INFINITY) s += p.y * __builtin_amdgcn_exp2f(p.x - mt);
      }
      const float r = mt + __builtin_amdgcn_logf(s);
      if (!isfinite(r)) report_nonfinite(g);
      lse2[u * M + rho] = r;
    }
  }
  if (SUM_FORMAT) {
    __syncthreads();
    if (threadIdx.x == 0) flag[u] = bad;
  }
}

// Row log2-sums from a caller's natural-log log-sum-exp, [L][B*w][Hq]
// (import), and back (export).  Row rho = q*G + gq of unit (l, b, h) is
// window query q of sequence b, query head h*G + gq.
template <bool IMPORT>
__global__ __launch_bounds__(256) void lse_io_kernel(Geo g, SeqTab st, const float* __restrict__ lse_in,
                                                      float* __restrict__ lse2,
                                                      float* __restrict__ lse_out) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int M = g.w * g.G;
  const int64_t u = unit_index(g, l, b, h);
  for (int rho = threadIdx.x; rho < M; rho += blockDim.x) {
    const int q = rho / g.G, gq = rho % g.G;
    const int64_t i = (((int64_t)l * g.B + b) * g.w + q) * ((int64_t)g.H * g.G) + h * g.G + gq;
    if (IMPORT) {
      const float x = lse_in[i];
      if (!isfinite(x)) report_nonfinite(g);
      lse2[u * M + rho] = x * kLog2e;
    } else {
      lse_out[i] = lse2[u * M + rho] * kLn2;
    }
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
    const size_t Mp = (size_t)score_nqt(M) * 32;
    const size_t q = Mp * (g.D + 8) * 2;
    const size_t nw = kScoreThreads / 64;
    const size_t red = nw * (Mp * 2 > (size_t)g.D ? Mp * 2 : (size_t)g.D) * 4;
    return (q > red ? q : red) + Mp * 8;
  }
  return (size_t)M * g.D * 4 + (size_t)M * 4 + 8 * 4 + (size_t)4 * g.D * 4;
}

template <int D, int NQT>
static certkv_status launch_mfma(const ScoreArgs& a, const SeqTab& st, int max_len,
                                 hipStream_t s) {
  const Geo& g = a.g;
  const int nkb = (max_len + a.keys_per_block - 1) / a.keys_per_block;
  const int nkb2 = (max_len + a.keys_per_block2 - 1) / a.keys_per_block2;
  dim3 grid(nkb, g.H * st.count, g.L);
  dim3 grid2(nkb2, g.H * st.count, g.L);
  size_t smem = score_smem_bytes(g, CERTKV_BF16);
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncSetAttribute((const void*)score_mfma_kernel<D, NQT, kPass1Sum>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    hipFuncSetAttribute((const void*)score_mfma_kernel<D, NQT, kPass1Max>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    hipFuncSetAttribute((const void*)score_pass2_kernel<D, NQT, true>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    hipFuncSetAttribute((const void*)score_pass2_kernel<D, NQT, false>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if constexpr (NQT <= 8) {
      hipFuncSetAttribute((const void*)score_pass2_w16_kernel<D, NQT, true>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      hipFuncSetAttribute((const void*)score_pass2_w16_kernel<D, NQT, false>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    }
    attr_set = true;
  }
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* k = static_cast<const uint16_t*>(a.k.ptr);
  if (a.lse_in) {
    CERTKV_LAUNCH("score_lse_import", lse_io_kernel<true>, dim3(g.H * st.count, g.L), dim3(256), 0,
                  s, g, st, a.lse_in, a.lse2, (float*)nullptr);
  } else {
    CERTKV_LAUNCH("score_pass1_mfma", (score_mfma_kernel<D, NQT, kPass1Sum>), grid,
                  dim3(kScoreThreads), smem, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                  a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block, a.nkb_max, a.part,
                  (const int32_t*)nullptr);
    CERTKV_LAUNCH("score_lse_combine", lse_combine_kernel<true>, dim3(g.H * st.count, g.L), dim3(256),
                  0, s, g, st, a.keys_per_block, a.nkb_max, (const float2*)a.part, a.lse2, a.flag, 0);
    // fallback for flagged units (returns at once for the others)
    CERTKV_LAUNCH("score_pass1_fallback", (score_mfma_kernel<D, NQT, kPass1Max>), grid,
                  dim3(kScoreThreads), smem, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                  a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block, a.nkb_max, a.part,
                  (const int32_t*)a.flag);
    CERTKV_LAUNCH("score_lse_fallback", lse_combine_kernel<false>, dim3(g.H * st.count, g.L),
                  dim3(256), 0, s, g, st, a.keys_per_block, a.nkb_max, (const float2*)a.part, a.lse2,
                  a.flag, 1);
  }
  if constexpr (NQT <= 8) {
    // windows of at most 256 rows: sixteen waves share the staged queries
    const size_t smem2 = P2Smem<D, NQT>::total;
    if (a.ksum)
      CERTKV_LAUNCH("score_pass2_mfma", (score_pass2_w16_kernel<D, NQT, true>), grid2,
                    dim3(kP2Threads), smem2, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                    a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block2, a.nkb2_max,
                    (const float*)a.lse2, a.scores, a.kpart);
    else
      CERTKV_LAUNCH("score_pass2_mfma", (score_pass2_w16_kernel<D, NQT, false>), grid2,
                    dim3(kP2Threads), smem2, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                    a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block2, a.nkb2_max,
                    (const float*)a.lse2, a.scores, (float*)nullptr);
  } else {
    if (a.ksum)
      CERTKV_LAUNCH("score_pass2_mfma", (score_pass2_kernel<D, NQT, true>), grid2,
                    dim3(kScoreThreads), smem, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                    a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block2, a.nkb2_max,
                    (const float*)a.lse2, a.scores, a.kpart);
    else
      CERTKV_LAUNCH("score_pass2_mfma", (score_pass2_kernel<D, NQT, false>), grid2,
                    dim3(kScoreThreads), smem, s, g, st, q, a.q.s_layer, a.q.s_token, a.q.s_head, k,
                    a.k.s_layer, a.k.s_token, a.k.s_head, a.keys_per_block2, a.nkb2_max,
                    (const float*)a.lse2, a.scores, (float*)nullptr);
  }
  if (a.ksum)
    CERTKV_LAUNCH("score_ksum_reduce", ksum_reduce_kernel, dim3(g.H * st.count, g.L), dim3(128), 0,
                  s, g, st, a.keys_per_block2, a.nkb2_max, (const float*)a.kpart, a.ksum);
  if (a.lse_out)
    CERTKV_LAUNCH("score_lse_export", lse_io_kernel<false>, dim3(g.H * st.count, g.L), dim3(256), 0,
                  s, g, st, (const float*)nullptr, a.lse2, a.lse_out);
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
  if (a.lse_in) {
    CERTKV_LAUNCH("score_lse_import", lse_io_kernel<true>, dim3(g.H * st.count, g.L), dim3(256), 0,
                  s, g, st, a.lse_in, a.lse2, (float*)nullptr);
  } else {
    CERTKV_LAUNCH("score_pass1_f32", (score_f32_kernel<D, false>), grid, dim3(256), smem, s, g, st,
                  q, a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token, a.k.s_head,
                  a.nkb_max, a.part, (const float*)nullptr, (float*)nullptr, (float*)nullptr);
    CERTKV_LAUNCH("score_lse_combine", lse_combine_kernel<false>, dim3(g.H * st.count, g.L),
                  dim3(256), 0, s, g, st, 256, a.nkb_max, (const float2*)a.part, a.lse2, a.flag, 0);
  }
  CERTKV_LAUNCH("score_pass2_f32", (score_f32_kernel<D, true>), grid, dim3(256), smem, s, g, st, q,
                a.q.s_layer, a.q.s_token, a.q.s_head, k, a.k.s_layer, a.k.s_token, a.k.s_head,
                a.nkb_max, (float2*)nullptr, (const float*)a.lse2, a.scores,
                a.ksum ? a.kpart : (float*)nullptr);
  if (a.ksum)
    CERTKV_LAUNCH("score_ksum_reduce", ksum_reduce_kernel, dim3(g.H * st.count, g.L), dim3(128), 0,
                  s, g, st, 256, a.nkb_max, (const float*)a.kpart, a.ksum);
  if (a.lse_out)
    CERTKV_LAUNCH("score_lse_export", lse_io_kernel<false>, dim3(g.H * st.count, g.L), dim3(256), 0,
                  s, g, st, (const float*)nullptr, a.lse2, a.lse_out);
  return CERTKV_OK;
}

template <int D>
static certkv_status dispatch_nqt(const ScoreArgs& a, const SeqTab& st, int max_len, hipStream_t s) {
  switch (score_nqt(a.g.w * a.g.G)) {
    case 1: return launch_mfma<D, 1>(a, st, max_len, s);
    case 2: return launch_mfma<D, 2>(a, st, max_len, s);
    case 4: return launch_mfma<D, 4>(a, st, max_len, s);
    case 8: return launch_mfma<D, 8>(a, st, max_len, s);
    default: return launch_mfma<D, 16>(a, st, max_len, s);
  }
}

certkv_status run_score(const ScoreArgs& a, const SeqTab& st, int max_len, hipStream_t s) {
  if (a.dtype == CERTKV_F32)
    return a.g.D == 128 ? launch_f32<128>(a, st, max_len, s) : launch_f32<64>(a, st, max_len, s);
  if (a.g.D == 128) return dispatch_nqt<128>(a, st, max_len, s);
  return dispatch_nqt<64>(a, st, max_len, s);
}

}  // namespace certkv
