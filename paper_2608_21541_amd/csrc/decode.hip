// Decode over the packed cache on gfx950.
//
// After the pass each head keeps its b_h real rows and one charged slot row
// (k*, v*) (Section 4.1); a later query attends over these rows as ordinary
// keys, the plain slot carrying no logit bias.  For the tq new queries of a
// sequence and KV head h, the M = tq * G query rows (row = t * G + g) attend
// over the unit's packed segment:
//   z_i = scale <q, k_i>,  out = sum_i softmax(z)_i v_i,  lse = log sum e^z.
//
// Split over keys: one workgroup per (unit, 1024-key chunk), the grid ordered
// unit-fastest so that the chunks of every unit are dispatched before the
// empty tail of the grid (which is sized for the longest segment the caller
// allows).  One wave per 32-row query tile; with fewer than four tiles the
// spare waves form groups that take alternate key tiles.  Key and value tiles
// of 32 rows are staged through LDS two at a time (16-byte range-checked
// loads prefetched into registers during the previous batch; the value tile
// is stored transposed, [dim][key]).  Per tile and wave:
//   S^T = K Q^T on v_mfma_f32_32x32x16_bf16 with the key tile as the A
//     operand, so lane (hh, c) holds query row c and 16 of the tile's keys;
//   online softmax in log2 units, the row maximum shared by the two lanes of
//     a row, the accumulators rescaled only when a row maximum grows by more
//     than 2^8 (weights stay below 2^8, the partial is unchanged);
//   O^T += V^T P^T on the same MFMA: P^T (B operand) comes straight from the
//     lane's registers, split into a bf16 high part and the bf16 of the
//     remainder (two MFMAs, about 16 bits of the fp32 weight), and V^T (A
//     operand) is two 8-byte reads of the transposed value tile along the
//     same key order.
// The chunk partials (reference max, sum, unnormalized output) are combined
// in split order by a second kernel (deterministic).
#include "stages.h"

namespace certkv {

constexpr int kDecKeys = 1024;  // keys per workgroup (one split)
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


// Workgroup shape: one wave per 32-row query tile, at least four waves; with
// fewer query tiles the KG = NW / NQT wave groups take different key tiles of
// a batch, each with its own softmax state and partial slot.
template <int NQT>
struct DecShape {
  static constexpr int NW = NQT < 4 ? 4 : NQT;  // waves per workgroup
  static constexpr int KG = NW / NQT;            // wave groups over the key tiles
};
constexpr int kDecBatch = 2;  // key tiles staged per iteration

// Two waves per SIMD: the register cap keeps the accumulators out of AGPRs
// without spilling (three waves would spill).
template <int D, int NQT>
__global__ __launch_bounds__(64 * DecShape<NQT>::NW)
__attribute__((amdgpu_waves_per_eu(2))) void decode_kernel(
    Geo g, int32_t tq, int32_t nsub, int32_t mp, const uint16_t* __restrict__ qn,
    int64_t q_sl, int64_t q_st, int64_t q_sh, const uint16_t* __restrict__ kp,
    const uint16_t* __restrict__ vp, const int64_t* __restrict__ poff,
    float* __restrict__ part_o, float2* __restrict__ part_ml) {
  constexpr int NW = DecShape<NQT>::NW;
  constexpr int KG = DecShape<NQT>::KG;
  constexpr int KS = D / 16;       // MFMA k-steps of S^T
  constexpr int HD = D / 2;        // dims per lane half in S^T
  constexpr int NDB = D / 32;      // 32-dim blocks of the output
  constexpr int RE = D + 8;        // padded LDS row of a key tile, bf16 elements
  constexpr int VT = kDecTile + 4; // padded LDS row of a transposed value tile
  constexpr int CH = D / 8;        // 16-byte chunks per row
  // the batch's key tiles [key][dim] and transposed value tiles [dim][key]
  __shared__ __align__(16) uint16_t k_lds[kDecBatch][kDecTile * RE];
  __shared__ __align__(16) uint16_t v_lds[kDecBatch][D * VT];

  // units along x, chunks along y: every unit's first chunks are dispatched
  // before any unit's later (possibly empty) ones
  const int64_t u = blockIdx.x;
  const int split = blockIdx.y;
  const int h = (int)(u % g.H);
  const int64_t lb = u / g.H;
  const int b = (int)(lb % g.B);
  const int l = (int)(lb / g.B);
  const int64_t p0 = poff[u];
  const int len = (int)(poff[u + 1] - p0);
  const int c0 = split * kDecKeys;
  if (c0 >= len) return;  // whole workgroup: this unit has fewer chunks
  const int c1 = min(len, c0 + kDecKeys);
  const int ntiles = (c1 - c0 + kDecTile - 1) / kDecTile;
  const int nbatch = (ntiles + kDecBatch - 1) / kDecBatch;
  const int M = tq * g.G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qt = wave % NQT;        // query tile of this wave
  const int kg = wave / NQT;        // its wave group over the key tiles
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  const int row = qt * 32 + c32;    // this lane's query row
  const float c2 = g.scale * kDecLog2e;

  // The query row as B fragments of S^T (zero for padding rows); lane half hh
  // owns the dims hh*HD .. hh*HD + HD - 1 (the contraction order is free).
  DecFrag qf[KS];
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

  // Cooperative staging of a batch in 16-byte chunks.  Within a tile, key
  // chunk e is row e / CH, chunk e % CH (coalesced rows); value chunk e is
  // key e % 32, chunk e / 32 (its transposed 2-byte writes then fall on
  // consecutive keys).  The loads go through range-checked buffers over the
  // unit's segment, unconditionally (a conditional load would make the
  // compiler wait for the whole prefetch at the branch join): rows past the
  // segment read as zero, rows past the chunk are masked from the softmax.
  const uint32_t seg_bytes = (uint32_t)len * D * 2u;
  const BufRsrc krs = make_rsrc(kp + p0 * D, seg_bytes);
  const BufRsrc vrs = make_rsrc(vp + p0 * D, seg_bytes);
  constexpr int NTHR = 64 * NW;
  constexpr int HCH = kDecBatch * kDecTile * CH;  // key (or value) chunks of a batch
  constexpr int PER = (HCH + NTHR - 1) / NTHR;    // of each per thread
  uint4 stage_k[PER], stage_v[PER];
  auto load_batch = [&](int tb) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = threadIdx.x + j * NTHR;
      if (HCH % NTHR == 0 || e < HCH) {
        const int tile = e / (kDecTile * CH), et = e % (kDecTile * CH);
        const int rk = et / CH, chk = et % CH;        // key tile: row-major chunks
        const int rv = et % kDecTile, chv = et / kDecTile;  // value tile: key-fastest
        const int tk = tb - c0 + tile * kDecTile;     // tile start within the chunk
        stage_k[j] = buf_load_u128(krs, ((uint32_t)(c0 + tk + rk) * D + chk * 8) * 2u);
        stage_v[j] = buf_load_u128(vrs, ((uint32_t)(c0 + tk + rv) * D + chv * 8) * 2u);
      }
    }
  };
  auto store_batch = [&]() {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = threadIdx.x + j * NTHR;
      if (HCH % NTHR == 0 || e < HCH) {
        const int tile = e / (kDecTile * CH), et = e % (kDecTile * CH);
        *reinterpret_cast<uint4*>(&k_lds[tile][(et / CH) * RE + (et % CH) * 8]) = stage_k[j];
        const int rv = et % kDecTile, chv = et / kDecTile;
        const uint16_t* x = reinterpret_cast<const uint16_t*>(&stage_v[j]);
#pragma unroll
        for (int q = 0; q < 8; ++q) v_lds[tile][(chv * 8 + q) * VT + rv] = x[q];
      }
    }
  };

  float m_run = -INFINITY, l_run = 0.f;
  dec_f32x16 O[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[db][v] = 0.f;

  // One key tile (LDS slot j, first key t0) for this wave's query tile.
  auto process_tile = [&](int j, int t0) {
    const uint16_t* kt = k_lds[j];
    const uint16_t* vt = v_lds[j];
    // S^T = K Q^T: lane (hh, c32) holds query row c32 and keys
    // 8*(v/4) + 4*hh + v%4 of the tile
    dec_f32x16 s;
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      DecFrag kf;
      kf.u = *reinterpret_cast<const uint4*>(kt + c32 * RE + hh * HD + ks * 8);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf.v, qf[ks].v, s, 0, 0, 0);
    }
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
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64)) * c2;
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
      for (int db = 0; db < NDB; ++db)
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
    // O^T += V^T P^T per 32-dim block; V^T lane (hh, c32) = dim 32 db + c32
    // over the same keys: keys 16 kk + 4 hh + 0..3 and 16 kk + 8 + 4 hh + 0..3
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        DecFrag vf;
        const uint16_t* vrow = vt + (32 * db + c32) * VT + 16 * kk + 4 * hh;
        const uint2 lo4 = *reinterpret_cast<const uint2*>(vrow);
        const uint2 hi4 = *reinterpret_cast<const uint2*>(vrow + 8);
        vf.u = make_uint4(lo4.x, lo4.y, hi4.x, hi4.y);
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, ph[kk].v, O[db], 0, 0, 0);
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pl[kk].v, O[db], 0, 0, 0);
      }
    }
  };

  load_batch(c0);
  store_batch();
  __syncthreads();
  for (int bi = 0; bi < nbatch; ++bi) {
    const int tb = c0 + bi * kDecBatch * kDecTile;
    if (bi + 1 < nbatch) load_batch(tb + kDecBatch * kDecTile);  // in flight meanwhile
    for (int j = kg; j < kDecBatch; j += KG) {
      const int t0 = tb + j * kDecTile;
      if (t0 < c1) process_tile(j, t0);
    }
    __syncthreads();  // the batch is consumed
    if (bi + 1 < nbatch) {
      store_batch();
      __syncthreads();
    }
  }

  // partials of this chunk and wave group: the row's (max, sum) and
  // unnormalized output (a group without tiles leaves max -inf, sum 0)
  const float l_row = l_run + __shfl_xor(l_run, 32, 64);
  const int64_t pr = ((int64_t)u * nsub + split * KG + kg) * mp + row;
  if (hh == 0) part_ml[pr] = make_float2(m_run, l_row);
  float* po = part_o + pr * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) po[32 * db + 8 * (v >> 2) + 4 * hh + (v & 3)] = O[db][v];
}

// Combine the chunk partials of each (unit, row): one workgroup per row, the
// partial slots dealt round-robin to groups of D/4 threads (four output dims
// per thread, 16-byte loads).  Each group folds its slots in order with an
// online maximum; the groups are then merged in group order through LDS, so
// the result does not depend on timing.  Slots of wave groups that saw no
// key carry max -inf and are skipped.
constexpr int kCombThreads = 256;

template <int D>
__global__ __launch_bounds__(kCombThreads) void decode_combine_kernel(
    Geo g, int32_t tq, int32_t nsub, int32_t kgroups, int32_t mp, const int64_t* __restrict__ poff,
    const float* __restrict__ part_o, const float2* __restrict__ part_ml, float* __restrict__ out,
    float* __restrict__ lse) {
  constexpr int C4 = D / 4;                // threads per slot row
  constexpr int S = kCombThreads / C4;     // slot groups
  __shared__ float4 acc_s[S][C4];
  __shared__ float2 ml_s[S];
  const int64_t u = blockIdx.x;
  const int row = blockIdx.y;
  const int sg = threadIdx.x / C4;
  const int c4 = threadIdx.x % C4;
  const int len = (int)(poff[u + 1] - poff[u]);
  const int nv = min(nsub, kgroups * ((len + kDecKeys - 1) / kDecKeys));
  if (len > (nsub / kgroups) * kDecKeys && row == 0 && threadIdx.x == 0) report_range(g);
  const int64_t base = (int64_t)u * nsub * mp + row;  // + slot * mp
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
  const int Hq = g.H * g.G;
  const int h = (int)(u % g.H);
  const int64_t lb = u / g.H;
  const int b = (int)(lb % g.B);
  const int l = (int)(lb / g.B);
  const int t = row / g.G, gq = row % g.G;
  const int64_t orow = ((int64_t)l * g.B * tq + (int64_t)b * tq + t) * Hq + h * g.G + gq;
  const float o = at / Lt;
  if (!isfinite(o)) report_nonfinite(g);
  out[orow * D + dd] = o;
  if (lse && dd == 0) lse[orow] = (mx + __builtin_amdgcn_logf(Lt)) * kDecLn2;
}

template <int D, int NQT>
static certkv_status launch_decode(const DecodeArgs& a, hipStream_t s) {
  const Geo& g = a.g;
  const int mp = NQT * 32;
  constexpr int KG = DecShape<NQT>::KG;
  const int nsub = a.nsplit * KG;
  dim3 grid((unsigned)a.U, a.nsplit);
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_packed);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_packed);
  CERTKV_LAUNCH("decode", (decode_kernel<D, NQT>), grid, dim3(64 * DecShape<NQT>::NW), 0, s, g,
                a.tq, nsub, mp, q, a.q.s_layer, a.q.s_token, a.q.s_head, kp, vp,
                a.packed_offsets, a.part_o, a.part_ml);
  const int M = a.tq * g.G;
  CERTKV_LAUNCH("decode_combine", decode_combine_kernel<D>, dim3((unsigned)a.U, (unsigned)M),
                dim3(kCombThreads), 0, s,
                g, a.tq, nsub, KG, mp, a.packed_offsets, (const float*)a.part_o,
                (const float2*)a.part_ml, a.out, a.lse);
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
  const int nqt = decode_nqt(tq * G);
  const int kg = nqt < 4 ? 4 / nqt : 1;  // wave groups per workgroup (DecShape)
  return (size_t)U * nsplit * kg * nqt * 32;
}

int decode_nsplit(int max_len) { return (max_len + kDecKeys - 1) / kDecKeys; }

}  // namespace certkv
