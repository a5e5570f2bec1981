// Dispersion curves c(b) = sqrt((m Q - |W|^2)_+) over the evicted suffix of
// the score order (the keys at ranks b..n-1), for b = 0..n-1, in fp64, with
// m, W and Q the suffix sums of a, a v and a |v|^2.
//
// One workgroup (16 waves) per unit walks the ranks from the top (rank n-1)
// down in chunks of 512.  Each half-wave owns 16 consecutive ranks of a chunk
// (sub-range s = 2 wave + half; s = 0 holds the highest ranks) and its lane i
// owns dims DP*i..DP*i+DP-1 (DP = d/32), so one wave step advances two ranks.
// Q is kept as per-lane parts (the lane's dims of sum a |v|^2), which add up
// to Q without a cross-lane reduction.  Per chunk:
//   phase 1  each half-wave forms the totals of its 16 rows: m, W (per dim)
//            and the lane parts of Q (with bf16 rows, each row's lane part
//            of |v|^2 stays in registers for phase 2);
//   carry    sub-range s starts from the chunk carry plus the totals of the
//            sub-ranges 0..s-1 (higher ranks), added in a fixed order
//            (deterministic);
//   phase 2  the half-wave walks its ranks top-down extending m, W and its
//            lane parts q; per rank each lane forms m q - |W|^2 over its dims
//            (its part of c^2) and leaves it in a wave-private LDS row; after
//            every 8 ranks each lane adds up one rank's parts of 8 lanes and
//            two lane exchanges complete the sums over the 32 lanes.
// The carry pass also forms the chunk carry plus every total, the carry of the
// next chunk, so a chunk needs two barriers (after phase 1 and after the carry
// pass) and a wave that finishes its walk early goes on to the next phase 1.
// The weights and row offsets of a wave's 32 ranks pass through a
// wave-private LDS table, so that each half reads those of its own rank.  The
// gathers are software-pipelined: once the walk has taken step r of chunk k,
// the row of step r of chunk k-1 is fetched into the same registers (one set
// of row registers, no copies), and the order/score entries of chunk k-2 are
// fetched at the top of chunk k.  Also emitted: sum_j (s_j)_+ v_j (the value
// total of the tail summary).
#include "stages.h"

namespace certkv {

constexpr int kCurveThreads = 1024;
constexpr int kCurveWaves = kCurveThreads / 64;
constexpr int kLPR = 32;                       // lanes per rank (a half-wave)
constexpr int kRPH = 16;                       // ranks per half-wave and chunk
constexpr int kSubs = 2 * kCurveWaves;         // sub-ranges per chunk
constexpr int kCurveChunk = kSubs * kRPH;      // 512 ranks

template <int DP, int RAW, bool BF16>
__device__ __forceinline__ void unpack_dims(const uint32_t (&raw)[RAW], float (&v)[DP]) {
#pragma unroll
  for (int t = 0; t < DP; ++t) {
    if (BF16)
      v[t] = (t & 1) ? bf16_hi(raw[t >> 1]) : bf16_lo(raw[t >> 1]);
    else
      v[t] = __uint_as_float(raw[t]);
  }
}

// RAW consecutive 32-bit words at byte offset `off` of the value slice.
template <int RAW>
__device__ __forceinline__ void load_words(BufRsrc r, uint32_t off, uint32_t (&dst)[RAW]) {
  if constexpr (RAW == 1) {
    dst[0] = buf_load_u32(r, off);
  } else if constexpr (RAW == 2) {
    const uint2 x = buf_load_u64(r, off);
    dst[0] = x.x;
    dst[1] = x.y;
  } else {
    static_assert(RAW == 4, "rows split into 4, 8 or 16 bytes per lane");
    const uint4 x = buf_load_u128(r, off);
    dst[0] = x.x;
    dst[1] = x.y;
    dst[2] = x.z;
    dst[3] = x.w;
  }
}

__device__ __forceinline__ double join_f64(uint32_t lo, uint32_t hi) {
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// x plus x of the lane 16 places away in the same half-wave.
// v_permlane16_swap of x with itself exchanges neighbouring rows of 16 lanes,
// leaving the lane's own value in one result and its partner's in the other.
__device__ __forceinline__ double sum_lane16(double x) {
  const uint64_t a = (uint64_t)__double_as_longlong(x);
  const auto r0 = __builtin_amdgcn_permlane16_swap((uint32_t)a, (uint32_t)a, false, false);
  const auto r1 = __builtin_amdgcn_permlane16_swap((uint32_t)(a >> 32), (uint32_t)(a >> 32), false,
                                                   false);
  return join_f64(r0[0], r1[0]) + join_f64(r0[1], r1[1]);
}

// The value x of the upper half-wave (lanes 0-31) and of the lower one
// (lanes 32-63), lane for lane, in every lane: v_permlane32_swap of x with
// itself leaves the upper half's values in its first result and the lower
// half's in its second.
__device__ __forceinline__ void halves(double x, double& top, double& bot) {
  const uint64_t a = (uint64_t)__double_as_longlong(x);
  const auto r0 = __builtin_amdgcn_permlane32_swap((uint32_t)a, (uint32_t)a, false, false);
  const auto r1 =
      __builtin_amdgcn_permlane32_swap((uint32_t)(a >> 32), (uint32_t)(a >> 32), false, false);
  top = join_f64(r0[0], r1[0]);
  bot = join_f64(r0[1], r1[1]);
}

// x of the lane 8 places along in the lane's row of 16 (DPP row rotation).
__device__ __forceinline__ double row_ror8(double x) {
  const uint64_t a = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)a, 0x128, 0xF, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(a >> 32), 0x128, 0xF, 0xF, false);
  return join_f64(lo, hi);
}

// A wave-uniform double, moved to scalar registers.
__device__ __forceinline__ double uniform_f64(double x) {
  const uint64_t a = (uint64_t)__double_as_longlong(x);
  return join_f64(__builtin_amdgcn_readfirstlane((uint32_t)a),
                  __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)));
}

// STAT: the curve statistic (0 centered, 1 uncentered, 2 tail mass), fixed at
// compile time so that the walk has no branch on it; -1 reads it from g.stat
// at run time (not launched: each statistic has its own instantiation).
template <int D, bool BF16, int STAT>
__global__ __launch_bounds__(kCurveThreads) void curves_kernel(
    Geo g, SeqTab st, const uint32_t* __restrict__ sorted_keys, const int32_t* __restrict__ perm,
    const double* __restrict__ ssum, const void* __restrict__ vc, int64_t v_sl, int64_t v_st,
    int64_t v_sh, float* __restrict__ curves, double* __restrict__ vsum) {
  constexpr int DP = D / kLPR;                 // dims per lane
  constexpr int E = BF16 ? 2 : 4;              // bytes per element
  constexpr int RAW = DP * E / 4;              // 32-bit words per lane per row
  constexpr int NR = DP + 2;                   // per-lane record: W (its dims), q, m
  // phase 1 keeps the lane parts of |v|^2 of its rows for the walk (bf16
  // rows; with fp32 rows the registers are not there and the walk recomputes)
  constexpr bool kKeepNorms = BF16;
  // Per lane of a half-wave: phase-1 totals of each wave (both halves), the
  // upper half's own totals, and the chunk carry (suffix sums above the
  // chunk; each column read and rewritten by one thread of the carry pass).
  // One record layout for all three keeps a single per-lane LDS address.
  __shared__ __align__(16) double tR[kCurveWaves][kLPR][NR];
  __shared__ __align__(16) double uR[kCurveWaves][kLPR][NR];
  __shared__ __align__(16) double cR[kLPR][NR];
  // per wave, by chunk parity: weights and row byte offsets (in 64-bit
  // slots) of its 32 ranks, entries 16 h + r: half h, step r
  __shared__ __align__(16) double wa[2][kCurveWaves][2 * kRPH];
  __shared__ __align__(16) uint64_t wo[2][kCurveWaves][2 * kRPH];
  // per lane: its parts of c^2 of 8 walk steps (rows padded to 9 doubles,
  // so that the writes of a step and the group reads are free of bank
  // conflicts)
  __shared__ __align__(16) double red[kCurveWaves][64][9];

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
  const int hf = lane >> 5;
  const int li = lane & (kLPR - 1);
  const double tot = ssum[u];
  // denominator of the weights, wave-uniform (kept in scalar registers)
  const double wden = uniform_f64(tot > 0.0 ? tot : (double)n);
  // Value slice of this (layer, head, sequence): rows of d elements, token
  // stride v_st; the host guarantees it spans less than 4 GiB.
  const BufRsrc vrs = make_rsrc(
      static_cast<const char*>(vc) + ((int64_t)l * v_sl + tok0 * v_st + (int64_t)h * v_sh) * E,
      (uint32_t)(((int64_t)(n - 1) * v_st + D) * E));
  const uint32_t vrow_bytes = (uint32_t)(v_st * E);
  const uint32_t vlane = (uint32_t)(li * DP * E);
  const BufRsrc krs = make_rsrc(sorted_keys + base, (uint32_t)n * 4u);
  const BufRsrc prs = make_rsrc(perm + base, (uint32_t)n * 4u);

  // rank of step r (0 = highest) of sub-range s of chunk k
  auto rank_of = [&](int k, int s, int r) {
    return k * kCurveChunk + (kSubs - 1 - s) * kRPH + kRPH - 1 - r;
  };
  // Order entry and radix key of the wave's rank li (half li / 16, step
  // li % 16) of chunk k.  Every lane loads (from a clamped, in-bounds rank) so
  // that no branch splits the pipelined loads; `valid` marks real ranks.
  auto fetch_meta = [&](int k, uint32_t& key, int& pos, bool& valid) {
    const int rk = rank_of(k, 2 * wave + (li >> 4), li & (kRPH - 1));
    valid = k >= 0 && rk < n;
    const uint32_t idx = (uint32_t)min(max(rk, 0), n - 1) * 4u;
    key = buf_load_u32(krs, idx);
    pos = (int)buf_load_u32(prs, idx);
  };
  // weight a = (s)_+ / sum (s)_+ (uniform when every score is zero); zero for
  // absent ranks, whose rows then add nothing
  auto weight = [&](uint32_t key, bool valid) -> double {
    if (!valid) return 0.0;
    const float s = desc_key_value(key);
    const double num = tot > 0.0 ? (s > 0.f ? (double)s : 0.0) : 1.0;
    return num / wden;
  };
  // Weights and row offsets of the wave's ranks of chunk k into its table
  // (row 0 stands in for absent ranks, whose weight is zero).  The table is
  // wave-private: the wave's later reads see these writes in program order.
  auto publish = [&](int k, uint32_t key, int pos, bool valid) {
    if (lane < 2 * kRPH) {
      wa[k & 1][wave][lane] = weight(key, valid);
      wo[k & 1][wave][lane] = (uint32_t)(valid ? min(max(pos, 0), n - 1) : 0) * vrow_bytes;
    }
  };
  // Value row of step r of the half-wave's ranks in table slot `sl`; rows are
  // clamped into the sequence, so every offset stays in the slice.
  auto fetch_row = [&](int sl, int r, uint32_t (&raw)[RAW]) {
    load_words<RAW>(vrs, (uint32_t)wo[sl][wave][hf * kRPH + r] + vlane, raw);
  };
  // weight of step r of this half-wave's ranks in table slot `sl`
  auto a_of = [&](int sl, int r) -> double {
    const double2 p = reinterpret_cast<const double2*>(&wa[sl][wave][hf * kRPH])[r >> 1];
    return (r & 1) ? p.y : p.x;
  };

  const int nch = (n + kCurveChunk - 1) / kCurveChunk;
  for (int i = threadIdx.x; i < kLPR * NR; i += kCurveThreads) (&cR[0][0])[i] = 0.0;

  uint32_t k_n1, k_n2;
  int p_n1, p_n2;
  bool ok_n1, ok_n2;
  uint32_t vcur[kRPH][RAW];
  {
    uint32_t k0;
    int p0;
    bool ok0;
    fetch_meta(nch - 1, k0, p0, ok0);
    fetch_meta(nch - 2, k_n1, p_n1, ok_n1);
    publish(nch - 1, k0, p0, ok0);
  }
  // The first chunk's rows one by one in step order, the order in which the
  // walk fetches them: with the same order on both paths into the loop, the
  // compiler's count of outstanding loads lets phase 1 wait for each row
  // separately rather than for all of them.
#pragma unroll
  for (int r = 0; r < kRPH; ++r) {
    fetch_row((nch - 1) & 1, r, vcur[r]);
    __builtin_amdgcn_sched_barrier(0);
  }

  for (int k = nch - 1; k >= 0; --k) {
    const int par = k & 1;
    // pipeline: order entries two chunks ahead; the table of chunk k-1 (slot
    // par ^ 1), whose rows the walk below fetches
    fetch_meta(k - 2, k_n2, p_n2, ok_n2);
    publish(k - 1, k_n1, p_n1, ok_n1);

    // phase 1: totals of each half's rows; the wave's totals (both halves)
    // and the upper half's own totals (for the lower half's carry)
    double vvs[kKeepNorms ? kRPH : 1];
    {
      double sW[DP], sq = 0.0, sm = 0.0;
#pragma unroll
      for (int t = 0; t < DP; ++t) sW[t] = 0.0;
#pragma unroll
      for (int r = 0; r < kRPH; ++r) {
        const double ar = a_of(par, r);
        float v[DP];
        unpack_dims<DP, RAW, BF16>(vcur[r], v);
        double vv = 0.0;
#pragma unroll
        for (int t = 0; t < DP; ++t) {
          const double vd = (double)v[t];
          sW[t] = fma(ar, vd, sW[t]);
          vv = fma(vd, vd, vv);
        }
        sq = fma(ar, vv, sq);
        sm += ar;
        if constexpr (kKeepNorms) vvs[r] = vv;
      }
      double tp[NR], bt[NR];
#pragma unroll
      for (int t = 0; t < DP; ++t) halves(sW[t], tp[t], bt[t]);
      halves(sq, tp[DP], bt[DP]);
      halves(sm, tp[DP + 1], bt[DP + 1]);
      if (hf == 0) {
#pragma unroll
        for (int t = 0; t < NR; ++t) {
          uR[wave][li][t] = tp[t];
          tR[wave][li][t] = tp[t] + bt[t];
        }
      }
    }
    __syncthreads();
    // Exclusive prefix over the waves of the totals, from the chunk carry, in
    // place: one (lane, field) column per thread, added in wave order.
    {
      constexpr int C = kLPR * NR;
      if (threadIdx.x < C) {
        const int col = threadIdx.x;
        double* t = &tR[0][0][0];
        // every total read first: one LDS round trip, then the additions
        double x[kCurveWaves];
#pragma unroll
        for (int w = 0; w < kCurveWaves; ++w) x[w] = t[w * C + col];
        double* cc = &cR[0][0] + col;
        double run = *cc;
#pragma unroll
        for (int w = 0; w < kCurveWaves; ++w) {
          t[w * C + col] = run;
          run += x[w];
        }
        // the chunk carry plus every total: the carry of the next chunk
        *cc = run;
      }
    }
    __syncthreads();
    // carry of this sub-range: chunk carry + totals of the waves above it
    // (+ the upper half of its own wave for the lower half)
    double W[DP], q, m;
    {
      const double* c = tR[wave][li];
#pragma unroll
      for (int t = 0; t < DP; ++t) W[t] = c[t];
      q = c[DP];
      m = c[DP + 1];
      if (hf) {
        const double* x = uR[wave][li];
#pragma unroll
        for (int t = 0; t < DP; ++t) W[t] += x[t];
        q += x[DP];
        m += x[DP + 1];
      }
    }
    // Opaque to the optimizer: keeps the rows packed between the phases
    // instead of holding their converted doubles.
#pragma unroll
    for (int r = 0; r < kRPH; ++r) {
#pragma unroll
      for (int e = 0; e < RAW; ++e) __asm__ volatile("" : "+v"(vcur[r][e]));
    }
    // phase 2: walk the ranks top-down.  Each lane's part of c^2 of step r
    // goes to slot r % 8 of its LDS row; after steps 7 and 15 the lanes with
    // li % 8 = j add up the parts of step j of the 8 lanes of their group
    // (li / 8), a row rotation by 8 lanes adds the neighbouring group and a
    // swap of 16-lane rows the other two.  c2r[h]: step 8 h + li % 8.
    double c2r[2];
#pragma unroll
    for (int r = 0; r < kRPH; ++r) {
      const double ar = a_of(par, r);
      float v[DP];
      unpack_dims<DP, RAW, BF16>(vcur[r], v);
      double vv = 0.0, w2 = 0.0;
#pragma unroll
      for (int t = 0; t < DP; ++t) {
        const double vd = (double)v[t];
        W[t] = fma(ar, vd, W[t]);
        w2 = fma(W[t], W[t], w2);
        if constexpr (!kKeepNorms) vv = fma(vd, vd, vv);
      }
      if constexpr (kKeepNorms) vv = vvs[r];
      m += ar;
      q = fma(ar, vv, q);
      // the lanes' parts sum to m Q - |W|^2 (centered), m Q (uncentered) or,
      // for the tail mass, m^2 (32 equal parts of m^2 / 32, exact), whose
      // square root is m
      const int stat = STAT >= 0 ? STAT : g.stat;
      double cur = stat == 0 ? fma(m, q, -w2) : stat == 1 ? m * q : (m * m) * (1.0 / kLPR);
      red[wave][lane][r & 7] = cur;
      // this row is spent: fetch row r of the next chunk into its registers
      fetch_row(par ^ 1, r, vcur[r]);
      if ((r & 7) == 7) {
        // Compiler barriers only: a wave's LDS accesses execute in order, so
        // the reads see every lane's writes of these 8 steps and the next
        // steps' writes follow the reads.
        __asm__ volatile("" ::: "memory");
        const double* col = &red[wave][hf * kLPR + (li >> 3) * 8][li & 7];
        double x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = col[i * 9];
        double s = ((x[0] + x[1]) + (x[2] + x[3])) + ((x[4] + x[5]) + (x[6] + x[7]));
        s += row_ror8(s);
        c2r[r >> 3] = sum_lane16(s);
        __asm__ volatile("" ::: "memory");
      }
    }
    const int r_mine = li & (kRPH - 1);
    const double c2 = (li & 8) ? c2r[1] : c2r[0];
    const int rk = rank_of(k, 2 * wave + hf, r_mine);
    if (li < kRPH && rk < n) {
      if (!isfinite(c2)) report_nonfinite(g);
      curves[base + rk] = (float)sqrt(c2 > 0.0 ? c2 : 0.0);
    }
    k_n1 = k_n2;
    p_n1 = p_n2;
    ok_n1 = ok_n2;
  }
  // the carry after the last chunk: the sums over every rank
  __syncthreads();
  if (vsum && wave == 0) {
    for (int i = lane; i < D; i += 64) vsum[u * D + i] = cR[i / DP][i % DP] * tot;
  }
}

template <int D, bool BF16>
static certkv_status launch_curves(const CurveArgs& a, const SeqTab& st, hipStream_t s) {
  const dim3 grid(a.g.H * st.count, a.g.L);
#define CERTKV_CURVES(STAT)                                                                        \
  CERTKV_LAUNCH("curves", (curves_kernel<D, BF16, STAT>), grid, dim3(kCurveThreads), 0, s, a.g, st, \
                a.sorted_keys, a.perm, a.ssum, a.v.ptr, a.v.s_layer, a.v.s_token, a.v.s_head,       \
                a.curves, a.vsum)
  if (a.g.stat == 0)
    CERTKV_CURVES(0);
  else if (a.g.stat == 1)
    CERTKV_CURVES(1);
  else
    CERTKV_CURVES(2);
#undef CERTKV_CURVES
  return CERTKV_OK;
}

certkv_status run_curves(const CurveArgs& a, const SeqTab& st, hipStream_t s) {
  if (a.dtype == CERTKV_BF16)
    return a.g.D == 128 ? launch_curves<128, true>(a, st, s) : launch_curves<64, true>(a, st, s);
  return a.g.D == 128 ? launch_curves<128, false>(a, st, s) : launch_curves<64, false>(a, st, s);
}

}  // namespace certkv
