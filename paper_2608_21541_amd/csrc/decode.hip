// Decode over the packed cache on gfx950.
//
// After the pass each head keeps its b_h real rows and one charged slot row
// (k*, v*) (Section 4.1); a later query attends over these rows as ordinary
// keys, the plain slot carrying no logit bias.  For the tq new queries of a
// sequence and KV head h, the M = tq * G query rows (row = t * G + g) attend
// over the unit's packed segment:
//   z_i = scale <q, k_i>,  out = sum_i softmax(z)_i v_i,  lse = log sum e^z.
//
// Split over keys: the work items are (unit, 4096-key chunk) pairs, listed on
// the device and taken in a fixed stride by a persistent grid of as many
// workgroups as stay resident.  A workgroup holds the unit's query tiles of
// 32 rows, one wave each; with fewer than four tiles, two or four waves share
// a tile and split its output dims.  Key and value tiles of 32 rows go from
// memory straight into LDS (wave-wide 16-byte LDS-DMA loads into a ring of
// five tile buffers, XOR-swizzled chunks, rows in natural order).  Per tile
// and wave:
//   S^T = K Q^T on v_mfma_f32_32x32x16_bf16 with the key tile as the A
//     operand, so lane (hh, c) holds query row c and 16 of the tile's keys;
//   online softmax in log2 units, the row maximum shared by the two lanes of
//     a row, the accumulators rescaled only when a row maximum grows by more
//     than 2^8 (weights stay below 2^8, the partial is unchanged);
//   O^T += V^T P^T on the same MFMA: P^T (B operand) comes straight from the
//     lane's registers, split into a bf16 high part and the bf16 of the
//     remainder (two MFMAs, about 16 bits of the fp32 weight), and V^T (A
//     operand) comes from transposing LDS reads of the key-major value tile
//     along the same key order.
// The chunk partials (reference max, sum, unnormalized output) are combined
// in split order by a second kernel (deterministic).
#include "stages.h"

namespace certkv {

constexpr int kDecKeys = 4096;  // keys per work item (one split)
constexpr int kDecTile = 32;    // keys per tile

typedef __bf16 dec_bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float dec_f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

union DecFrag {
  uint4 u;
  uint16_t h[8];
  dec_bf16x8 v;
};

constexpr float kDecLog2e = 1.4426950408889634f;
constexpr float kDecLn2 = 0.6931471805599453f;
constexpr float kDecSlack = 8.f;  // log2 growth of the row maximum absorbed without rescaling

typedef __bf16 dec_bf16x2 __attribute__((ext_vector_type(2)));
typedef float dec_f32x2 __attribute__((ext_vector_type(2)));

// Two floats to bf16 (round to nearest even), a in the low half.
__device__ __forceinline__ uint32_t dec_pack_bf16(float a, float b) {
  const dec_bf16x2 h = __builtin_convertvector((dec_f32x2){a, b}, dec_bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}


// Workgroup shape: every wave takes one 32-row query tile and all keys; with
// fewer than four query tiles, DS waves share a query tile and split the
// output dims (each computes the tile's scores and softmax, and P V for its
// D / DS dims), down to 32 dims per wave.
template <int D, int NQT>
struct DecShape {
  static constexpr int DS0 = NQT >= 4 ? 1 : 4 / NQT;
  static constexpr int DS = DS0 < D / 32 ? DS0 : D / 32;  // dim splits per query tile
  static constexpr int NW = NQT * DS;                      // waves per workgroup
  static constexpr int NDBW = D / 32 / DS;                 // 32-dim blocks per wave
};

// LDS pipeline: a stage is one key tile (K and V); NBUF stage buffers, up to
// kDecLdsBytes and at most five (two workgroups per compute unit).
constexpr int kDecLdsBytes = 80 * 1024;
template <int D>
struct DecPipe {
  static constexpr int STAGE_BYTES = 2 * kDecTile * D * 2;
  static constexpr int NB0 = kDecLdsBytes / STAGE_BYTES;
  static constexpr int NBUF = NB0 > 5 ? 5 : NB0;
  static_assert(NBUF >= 3, "three stage buffers at least");
};

// LDS layout of a stage: [tile][K, V][32 rows][D/8 chunks of 16 bytes], rows
// in natural (key-major) order.  Chunks are XOR-swizzled within a row so that
// both fragment reads are free of bank conflicts: the key-tile read (one
// 16-byte chunk per lane, 16 consecutive rows per pass) and the transposing
// value-tile read (8 bytes per lane, four consecutive rows and eight
// consecutive 32-byte segments per half-wave).  The map is an involution:
// the slot of chunk c is c ^ f(r) and the chunk in slot s is s ^ f(r).
template <int D>
__device__ __forceinline__ int dec_swz_k(int r, int c) {
  return c ^ ((D == 128 ? r : (r >> 1)) & (D / 8 - 1));
}
template <int D>
__device__ __forceinline__ int dec_swz_v(int r, int c) {
  return c ^ (D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1));
}

// One wave-wide 16-byte load straight into LDS: lane L's 16 bytes from src
// land at LDS byte address lds + 16 L (lds wave-uniform, through M0).  Issued
// as inline assembly so that the compiler does not treat the load as a
// pending LDS write (which would make it wait for every load in flight at
// each barrier); the caller waits for it with dec_wait_vm0 before the
// barrier that publishes the stage.
__device__ __forceinline__ void dec_dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}

// Wait until at most N vector-memory accesses of this wave are in flight
// (the other counters at their maximum; a builtin, so the compiler's own
// bookkeeping of outstanding loads sees it).
template <int N>
__device__ __forceinline__ void dec_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void dec_wait_vm0() { dec_wait_vm<0>(); }

// dec_wait_vm<PER * n> for a wave-uniform n in [0, NMAX].
template <int PER, int NMAX>
__device__ __forceinline__ void dec_wait_stages(int n) {
  if constexpr (NMAX == 0) {
    dec_wait_vm<0>();
  } else {
    if (n >= NMAX)
      dec_wait_vm<PER * NMAX>();
    else
      dec_wait_stages<PER, NMAX - 1>(n);
  }
}

__device__ __forceinline__ uint32_t dec_lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

typedef short dec_s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) dec_s16x4 dec_lds_s16x4;

// The work items of a decode: every (unit, chunk) pair whose chunk starts
// inside the unit's segment (at most nsplit chunks per unit), unit-major.  One
// workgroup scans the per-unit chunk counts in rounds of kItemThreads units.
constexpr int kItemThreads = 1024;
__global__ __launch_bounds__(kItemThreads) void decode_items_kernel(
    int64_t U, int32_t nsplit, const int64_t* __restrict__ poff, int2* __restrict__ items,
    int32_t* __restrict__ count) {
  __shared__ int scan[kItemThreads];
  const int t = threadIdx.x;
  int base = 0;  // items of the earlier rounds
  for (int64_t u0 = 0; u0 < U; u0 += kItemThreads) {
    const int64_t u = u0 + t;
    int n = 0;
    if (u < U) {
      const int64_t len = poff[u + 1] - poff[u];
      n = (int)min((int64_t)nsplit, (len + kDecKeys - 1) / kDecKeys);
    }
    scan[t] = n;
    __syncthreads();
    for (int d = 1; d < kItemThreads; d <<= 1) {  // inclusive scan
      const int x = t >= d ? scan[t - d] : 0;
      __syncthreads();
      scan[t] += x;
      __syncthreads();
    }
    const int start = base + scan[t] - n;
    for (int k = 0; k < n; ++k) items[start + k] = make_int2((int)u, k);
    base += scan[kItemThreads - 1];
    __syncthreads();  // scan[] is rewritten by the next round
  }
  if (t == 0) *count = base;
}

// Two waves per SIMD: the register cap keeps the accumulators out of AGPRs.
template <int D, int NQT>
__global__ __launch_bounds__((64 * DecShape<D, NQT>::NW))
__attribute__((amdgpu_waves_per_eu(2))) void decode_kernel(
    Geo g, const int2* __restrict__ items, const int32_t* __restrict__ item_count,
    int32_t tq, int32_t nsplit, int32_t mp,
    const uint16_t* __restrict__ qn, int64_t q_sl, int64_t q_st, int64_t q_sh,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
    const int64_t* __restrict__ poff, float* __restrict__ part_o, float2* __restrict__ part_ml) {
  constexpr int NW = DecShape<D, NQT>::NW;
  constexpr int NDBW = DecShape<D, NQT>::NDBW;
  constexpr int NBUF = DecPipe<D>::NBUF;
  constexpr int KS = D / 16;       // MFMA k-steps of S^T
  constexpr int HD = D / 2;        // dims per lane half in S^T
  constexpr int CH = D / 8;        // 16-byte chunks per row
  constexpr int TILE = kDecTile * D;          // bf16 elements of one K (or V) tile
  constexpr int TILE_CH = kDecTile * CH;      // its 16-byte chunks
  constexpr int NINS = 2 * TILE_CH / 64;      // wave-wide 16-byte loads per stage
  constexpr int PERW = NINS >= NW ? NINS / NW : 1;  // of them per wave (or none)
  static_assert((NINS % NW == 0 || NINS < NW) && TILE_CH % 64 == 0, "stage split");
  __shared__ __align__(16) uint16_t lds[NBUF][2][TILE];

  // A persistent grid over the work items (unit, chunk), taken in a fixed
  // stride: consecutive chunks of a long segment go to different workgroups.
  const int nitems = *item_count;
  for (int item = blockIdx.x; item < nitems; item += gridDim.x) {
  const int2 it = items[item];
  const int64_t u = it.x;
  const int split = it.y;
  const int h = (int)(u % g.H);
  const int64_t lb = u / g.H;
  const int b = (int)(lb % g.B);
  const int l = (int)(lb / g.B);
  const int64_t p0 = poff[u];
  const int len = (int)(poff[u + 1] - p0);
  const int c0 = split * kDecKeys;
  if (c0 >= len) continue;  // whole workgroup: this unit has fewer chunks
  const int c1 = min(len, c0 + kDecKeys);
  const int ntiles = (c1 - c0 + kDecTile - 1) / kDecTile;
  const int M = tq * g.G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qt = wave % NQT;        // query tile of this wave
  const int dsi = wave / NQT;       // its share of the output dims
  const int db0 = dsi * NDBW;       // first 32-dim block of that share
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  const int row = qt * 32 + c32;    // this lane's query row
  const float c2 = g.scale * kDecLog2e;

  // A stage goes from memory straight into LDS: wave-wide 16-byte loads, lane
  // L of load n filling chunk slot 64 n + L of the stage.  The chunk a slot
  // holds is chosen by the swizzle; rows past the segment are clamped to its
  // last row (their keys are masked, so they only ever meet zero weights).
  const uint16_t* kseg = kp + p0 * D;
  const uint16_t* vseg = vp + p0 * D;
  auto issue_stage = [&](int st) {
#pragma unroll
    for (int i = 0; i < PERW; ++i) {
      const int n = wave * PERW + i;
      const int kv = n / (TILE_CH / 64);                    // uniform over the wave
      if (n < NINS) {
        const int pos = (n % (TILE_CH / 64)) * 64 + lane;   // slot within the tile
        const int r = pos / CH;
        const int chunk = kv ? dec_swz_v<D>(r, pos % CH) : dec_swz_k<D>(r, pos % CH);
        const int key = min(c0 + st * kDecTile + r, len - 1);
        const uint16_t* src = (kv ? vseg : kseg) + (int64_t)key * D + chunk * 8;
        dec_dma16(src, dec_lds_addr(&lds[st % NBUF][kv][(n % (TILE_CH / 64)) * 512]));
      }
    }
  };

  DecFrag qf[KS];
  float m_run = -INFINITY, l_run = 0.f;
  dec_f32x16 O[NDBW];  // O^T of the wave's 32-dim blocks db0 ..
#pragma unroll
  for (int db = 0; db < NDBW; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[db][v] = 0.f;

  // S^T = K Q^T of the key tile in stage buffer sb: lane (hh, c32) holds
  // query row c32 and keys 8*(v/4) + 4*hh + v%4 of the tile.
  auto score_tile = [&](int sb) {
    const uint16_t* kt = lds[sb][0];
    dec_f32x16 s;
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      DecFrag kf;
      kf.u = *reinterpret_cast<const uint4*>(kt + c32 * D +
                                             dec_swz_k<D>(c32, hh * (CH / 2) + ks) * 8);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf.v, qf[ks].v, s, 0, 0, 0);
    }
    return s;
  };

  // Softmax and O^T += V^T P^T of the tile (first key t0) whose scores are s.
  auto finish_tile = [&](int sb, int t0, dec_f32x16 s) {
    const uint16_t* vt = lds[sb][1];
    // Online softmax of the row in log2 units (z = c2 * s, c2 > 0, so the
    // maximum is taken on the raw products).  Keys past the chunk occur only
    // in its last tile.
    if (t0 + kDecTile > c1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = t0 + 8 * (v >> 2) + 4 * hh + (v & 3);
        s[v] = key < c1 ? s[v] : -INFINITY;
      }
    }
    float mt = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mt = fmaxf(mt, s[v]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt),
                                                       false, false);
      mt = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c2;
    }
    // Lazy rescaling: the reference maximum m_run moves only when some row of
    // the wave would otherwise see a weight above 2^kDecSlack; the weights
    // exp2(z - m_run) then stay below 2^kDecSlack and the partial (m_run,
    // l_run, O) is the same quantity for any reference.
    if (__builtin_amdgcn_ballot_w64(mt > m_run + kDecSlack) != 0) {
      const float mnew = fmaxf(m_run, mt);
      const float alpha = __builtin_amdgcn_exp2f(m_run - mnew);
      m_run = mnew;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDBW; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) O[db][v] *= alpha;
    }
    // P^T fragments: k-step kk takes the lane's values v = 8 kk .. 8 kk + 7,
    // i.e. keys 16 kk + 8 (i/4) + 4 hh + i%4 for k-slot 8 hh + i; each weight
    // is the bf16 (round to nearest even) of p plus the bf16 of p - hi.
    DecFrag ph[2], pl[2];
#pragma unroll
    for (int v = 0; v < 16; v += 2) {
      const float p0 = __builtin_amdgcn_exp2f(fmaf(s[v], c2, -m_run));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(s[v + 1], c2, -m_run));
      l_run += p0 + p1;
      const uint32_t hi = dec_pack_bf16(p0, p1);
      const float r0 = p0 - __uint_as_float(hi << 16);
      const float r1 = p1 - __uint_as_float(hi & 0xffff0000u);
      reinterpret_cast<uint32_t*>(&ph[v >> 3].u)[(v & 7) >> 1] = hi;
      reinterpret_cast<uint32_t*>(&pl[v >> 3].u)[(v & 7) >> 1] = dec_pack_bf16(r0, r1);
    }
    // O^T += V^T P^T per 32-dim block.  V^T (A operand): lane (hh, c32) needs
    // dim 32 db + c32 at the keys of its k-slots.  A transposing read serves
    // them from the key-major tile: in each group of 16 lanes, lane a
    // addresses key 16 kk + 8 rd + 4 hh + a/4 at dims 4 (a%4) .. 4 (a%4) + 3
    // of its group's 16 dims, and lane i receives dim i of keys
    // 16 kk + 8 rd + 4 hh + 0..3, which are its k-slots 4 rd .. 4 rd + 3.
    const int a = c32 & 15;
    const int vdim = 16 * (c32 >> 4) + 4 * (a & 3);  // + 32 db
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int db = 0; db < NDBW; ++db) {
        DecFrag vf;
#pragma unroll
        for (int rd = 0; rd < 2; ++rd) {
          const int r = 16 * kk + 8 * rd + 4 * hh + (a >> 2);
          const int dim = 32 * (db0 + db) + vdim;
          const uint16_t* src = vt + r * D + dec_swz_v<D>(r, dim >> 3) * 8 + (dim & 7);
          const dec_s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (dec_lds_s16x4*)(__attribute__((address_space(3))) uint16_t*)src);
          reinterpret_cast<uint2*>(&vf.u)[rd] = __builtin_bit_cast(uint2, x);
        }
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, ph[kk].v, O[db], 0, 0, 0);
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pl[kk].v, O[db], 0, 0, 0);
      }
    }
  };

  // Stage 0 and the query fragments are awaited together; then stages up to
  // NBUF - 2 ahead of the one consumed are in flight.  Before stage st each
  // wave waits until its own loads of st have landed (loads complete in
  // order, so those of the later stages already issued may stay in flight);
  // the barrier then publishes stage st and certifies that every wave is done
  // with stage st - 1, whose buffer the loads of stage st + NBUF - 1
  // overwrite.
  issue_stage(0);
  // The query row as B fragments of S^T (zero for padding rows); lane half hh
  // owns the dims hh*HD .. hh*HD + HD - 1 (the contraction order is free).
  if (row < M) {
    const int t = row / g.G, gq = row % g.G;
    const uint4* src = reinterpret_cast<const uint4*>(
        qn + (int64_t)l * q_sl + (int64_t)(b * tq + t) * q_st + (int64_t)(h * g.G + gq) * q_sh +
        hh * HD);
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s].u = src[s];
  } else {
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s].u = make_uint4(0u, 0u, 0u, 0u);
  }

  dec_wait_vm0();
  for (int st = 1; st < NBUF - 1 && st < ntiles; ++st) issue_stage(st);
  for (int st = 0; st < ntiles; ++st) {
    dec_wait_stages<PERW, NBUF - 2>(min(NBUF - 2, ntiles - 1 - st));
    __syncthreads();
    if (st + NBUF - 1 < ntiles) issue_stage(st + NBUF - 1);
    finish_tile(st % NBUF, c0 + st * kDecTile, score_tile(st % NBUF));
  }
  // partials of this chunk: the row's (max, sum), from the first wave of the
  // query tile (every wave of it holds the same), and the unnormalized output
  // of each wave's dims
  const float l_row = l_run + __shfl_xor(l_run, 32, 64);
  const int64_t pr = ((int64_t)u * nsplit + split) * mp + row;
  if (dsi == 0 && hh == 0) part_ml[pr] = make_float2(m_run, l_row);
  float* po = part_o + pr * D;
#pragma unroll
  for (int db = 0; db < NDBW; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      po[32 * (db0 + db) + 8 * (v >> 2) + 4 * hh + (v & 3)] = O[db][v];
  __syncthreads();  // every wave is done with the stage buffers of this item
  }
}

// Combine the chunk partials of each (unit, row): one workgroup per row, the
// partial slots dealt round-robin to groups of D/4 threads (four output dims
// per thread, 16-byte loads).  Each group folds its slots in order with an
// online maximum; the groups are then merged in group order through LDS, so
// the result does not depend on timing.
constexpr int kCombThreads = 256;

// With clustered tail summaries (CL), the m cluster terms n_g e^{lbar_g}
// (lbar_g = scale <q, kbar_g>) and n_g e^{lbar_g} vbar_g join the kept rows'
// sums (the ratio estimator of the clustered-summary bound), and the row's
// runtime certificate is evaluated from the stored summaries: with r_g =
// scale |q| R_g and zeta_g = n_g e^{lbar_g} / Zhat,
//   D_Z / Zhat = sum_g (e^r_g - 1) e^r_g zeta_g,
//   D_N / Zhat = sum_g e^r_g zeta_g ((e^r_g - 1) |vbar_g| + rho_g),
//   V' = max(max kept |v|, max_g |vbar_g| + rho_g),
// and |Ohat - O| <= 3 (D_N + V' D_Z) / Zhat when D_Z <= Zhat / 3 (else the
// bound is infinite).
template <int D, bool CL>
__global__ __launch_bounds__(kCombThreads) void decode_combine_kernel(
    Geo g, int32_t tq, int32_t nsplit, int32_t mp, const int64_t* __restrict__ poff,
    const float* __restrict__ part_o, const float2* __restrict__ part_ml, float* __restrict__ out,
    float* __restrict__ lse, DecodeClusters cl, const uint16_t* __restrict__ qn, int64_t q_sl,
    int64_t q_st, int64_t q_sh) {
  constexpr int kMaxCl = 64;
  __shared__ float zc_s[CL ? kMaxCl : 1], vn_s[CL ? kMaxCl : 1];
  __shared__ float qn_s;
  constexpr int C4 = D / 4;                // threads per slot row
  constexpr int S = kCombThreads / C4;     // slot groups
  __shared__ float4 acc_s[S][C4];
  __shared__ float2 ml_s[S];
  const int64_t u = blockIdx.x;
  const int row = blockIdx.y;
  const int sg = threadIdx.x / C4;
  const int c4 = threadIdx.x % C4;
  const int len = (int)(poff[u + 1] - poff[u]);
  const int nv = min(nsplit, (len + kDecKeys - 1) / kDecKeys);
  if (len > nsplit * kDecKeys && row == 0 && threadIdx.x == 0) report_range(g);
  const int64_t base = (int64_t)u * nsplit * mp + row;  // + slot * mp
  float m = -INFINITY, L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  auto fold = [&](float2 ml, float4 o) {
    if (ml.x == -INFINITY) return;
    if (ml.x > m) {
      const float a = __builtin_amdgcn_exp2f(m - ml.x);  // 0 while m is -inf
      L *= a;
      acc.x *= a; acc.y *= a; acc.z *= a; acc.w *= a;
      m = ml.x;
    }
    const float w = __builtin_amdgcn_exp2f(ml.x - m);
    L += ml.y * w;
    acc.x += o.x * w; acc.y += o.y * w; acc.z += o.z * w; acc.w += o.w * w;
  };
  int sp = sg;
  for (; sp + 3 * S < nv; sp += 4 * S) {  // four slots in flight
    float2 ml[4];
    float4 o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t pr = base + (int64_t)(sp + i * S) * mp;
      ml[i] = part_ml[pr];
      o[i] = reinterpret_cast<const float4*>(part_o + pr * D)[c4];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) fold(ml[i], o[i]);
  }
  for (; sp < nv; sp += S) {
    const int64_t pr = base + (int64_t)sp * mp;
    fold(part_ml[pr], reinterpret_cast<const float4*>(part_o + pr * D)[c4]);
  }
  acc_s[sg][c4] = acc;
  if (c4 == 0) ml_s[sg] = make_float2(m, L);
  const int Hq = g.H * g.G;
  const int h = (int)(u % g.H);
  const int64_t lb = u / g.H;
  const int b = (int)(lb % g.B);
  const int l = (int)(lb / g.B);
  const int t = row / g.G, gq = row % g.G;
  const int64_t orow = ((int64_t)l * g.B * tq + (int64_t)b * tq + t) * Hq + h * g.G + gq;
  const float c2 = g.scale * kDecLog2e;
  if (CL && threadIdx.x < cl.m) {
    // cluster logits in log2 units (with log2 n_g) and value norms
    const int gi = threadIdx.x;
    const uint16_t* qr = qn + (int64_t)l * q_sl + (int64_t)(b * tq + t) * q_st +
                         (int64_t)(h * g.G + gq) * q_sh;
    const uint16_t* kr = cl.kbar + (u * cl.m + gi) * D;
    const uint16_t* vr = cl.vbar + (u * cl.m + gi) * D;
    float dot = 0.f, vv = 0.f, qq = 0.f;
    for (int e = 0; e < D; ++e) {
      const float qe = bf16_to_f32(qr[e]);
      dot = fmaf(qe, bf16_to_f32(kr[e]), dot);
      const float ve = bf16_to_f32(vr[e]);
      vv = fmaf(ve, ve, vv);
      qq = fmaf(qe, qe, qq);
    }
    const int cnt = cl.count[u * cl.m + gi];
    zc_s[gi] = cnt > 0 ? dot * c2 + __builtin_amdgcn_logf((float)cnt) : -INFINITY;
    vn_s[gi] = sqrtf(vv);
    if (gi == 0) qn_s = sqrtf(qq);
  }
  __syncthreads();
  if (threadIdx.x >= D) return;
  const int dd = threadIdx.x;
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < S; ++k) mx = fmaxf(mx, ml_s[k].x);
  float Lt = 0.f, at = 0.f;
#pragma unroll
  for (int k = 0; k < S; ++k) {
    const float2 mk = ml_s[k];
    if (mk.x == -INFINITY) continue;
    const float w = __builtin_amdgcn_exp2f(mk.x - mx);
    Lt += mk.y * w;
    at += reinterpret_cast<const float*>(&acc_s[k][0])[dd] * w;
  }
  if (CL) {
    float mc = mx;
    for (int gi = 0; gi < cl.m; ++gi) mc = fmaxf(mc, zc_s[gi]);
    const float a = mx == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mx - mc);
    const float Ls = Lt * a;  // the kept rows' share, relative to 2^mc
    Lt = Ls;
    at *= a;
    for (int gi = 0; gi < cl.m; ++gi) {
      if (zc_s[gi] == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(zc_s[gi] - mc);
      Lt += w;
      at = fmaf(w, bf16_to_f32(cl.vbar[(u * cl.m + gi) * D + dd]), at);
    }
    mx = mc;
    if (dd == 0 && cl.bound) {
      const double rq = (double)g.scale * (double)qn_s;
      double dz = 0.0, dn = 0.0, vmax = (double)cl.vmax_kept[u];
      for (int gi = 0; gi < cl.m; ++gi)
        if (zc_s[gi] != -INFINITY) vmax = fmax(vmax, (double)vn_s[gi] + (double)cl.rv[u * cl.m + gi]);
      for (int gi = 0; gi < cl.m; ++gi) {
        if (zc_s[gi] == -INFINITY) continue;
        const double zeta = exp2((double)zc_s[gi] - (double)mc) / (double)Lt;
        const double er = exp(rq * (double)cl.rk[u * cl.m + gi]);
        dz += (er - 1.0) * er * zeta;
        dn += er * zeta * ((er - 1.0) * (double)vn_s[gi] + (double)cl.rv[u * cl.m + gi]);
      }
      cl.bound[orow] = dz <= 1.0 / 3.0 ? (float)(3.0 * (dn + vmax * dz)) : INFINITY;
    }
  }
  const float o = at / Lt;
  if (!isfinite(o)) report_nonfinite(g);
  out[orow * D + dd] = o;
  if (lse && dd == 0) lse[orow] = (mx + __builtin_amdgcn_logf(Lt)) * kDecLn2;
}

template <int D, int NQT>
static certkv_status launch_decode(const DecodeArgs& a, hipStream_t s) {
  const Geo& g = a.g;
  const int mp = NQT * 32;
  // as many workgroups as stay resident at once (the occupancy query is made
  // once per device and kernel instance)
  constexpr int NT = 64 * DecShape<D, NQT>::NW;
  static std::atomic<int> per_cu[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CERTKV_EHIP;
  int nb = per_cu[dev].load(std::memory_order_relaxed);
  if (nb == 0) {
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, decode_kernel<D, NQT>, NT, 0) !=
        hipSuccess)
      return CERTKV_EHIP;
    nb = nb > 0 ? nb : 1;
    per_cu[dev].store(nb, std::memory_order_relaxed);
  }
  const int cus = device_cus(dev);
  if (cus <= 0) return CERTKV_EHIP;
  const int64_t max_items = a.U * a.nsplit;
  const int64_t want = (int64_t)cus * nb;
  const unsigned grid = (unsigned)(max_items < want ? max_items : want);
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_packed);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_packed);
  CERTKV_LAUNCH("decode_items", decode_items_kernel, dim3(1), dim3(kItemThreads), 0, s, a.U,
                a.nsplit, a.packed_offsets, a.items, a.item_count);
  CERTKV_LAUNCH("decode", (decode_kernel<D, NQT>), dim3(grid), dim3(NT), 0, s, g, a.items,
                a.item_count, a.tq, a.nsplit, mp, q, a.q.s_layer, a.q.s_token, a.q.s_head, kp, vp,
                a.packed_offsets, a.part_o, a.part_ml);
  const int M = a.tq * g.G;
  if (a.cl.m > 0)
    CERTKV_LAUNCH("decode_combine", (decode_combine_kernel<D, true>),
                  dim3((unsigned)a.U, (unsigned)M), dim3(kCombThreads), 0, s, g, a.tq, a.nsplit, mp,
                  a.packed_offsets, (const float*)a.part_o, (const float2*)a.part_ml, a.out, a.lse,
                  a.cl, q, a.q.s_layer, a.q.s_token, a.q.s_head);
  else
    CERTKV_LAUNCH("decode_combine", (decode_combine_kernel<D, false>),
                  dim3((unsigned)a.U, (unsigned)M), dim3(kCombThreads), 0, s, g, a.tq, a.nsplit, mp,
                  a.packed_offsets, (const float*)a.part_o, (const float2*)a.part_ml, a.out, a.lse,
                  a.cl, q, a.q.s_layer, a.q.s_token, a.q.s_head);
  return CERTKV_OK;
}

template <int D>
static certkv_status launch_decode_d(const DecodeArgs& a, hipStream_t s) {
  switch (decode_nqt(a.tq * a.g.G)) {
    case 1: return launch_decode<D, 1>(a, s);
    case 2: return launch_decode<D, 2>(a, s);
    case 4: return launch_decode<D, 4>(a, s);
    case 8: return launch_decode<D, 8>(a, s);
    default: return launch_decode<D, 16>(a, s);
  }
}

certkv_status run_decode(const DecodeArgs& a, hipStream_t s) {
  return a.g.D == 128 ? launch_decode_d<128>(a, s) : launch_decode_d<64>(a, s);
}

size_t decode_partial_rows(int64_t U, int nsplit, int tq, int G) {
  return (size_t)U * nsplit * decode_nqt(tq * G) * 32;
}

int decode_nsplit(int max_len) { return (max_len + kDecKeys - 1) / kDecKeys; }

}  // namespace certkv
