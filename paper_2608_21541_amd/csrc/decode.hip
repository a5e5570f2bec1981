// Decode over the packed cache on gfx950.
//
// After the pass each head keeps its b_h real rows and one charged slot row
// (k*, v*) (Section 4.1); a later query attends over these rows as ordinary
// keys, the plain slot carrying no logit bias.  For the tq new queries of a
// sequence and KV head h, the M = tq * G query rows (row = t * G + g) attend
// over the unit's packed segment:
//   z_i = scale <q, k_i>,  out = sum_i softmax(z)_i v_i,  lse = log sum e^z.
//
// Split over keys: one workgroup per (unit, 1024-key chunk), one wave per
// 32-row query tile.  Key and value tiles of 32 rows are staged through LDS
// (coalesced 16-byte loads, prefetched into registers one tile ahead,
// double-buffered).  Per tile and wave:
//   S^T = K Q^T on v_mfma_f32_32x32x16_bf16 with the key tile as the A
//     operand, so lane (hh, c) holds query row c and 16 of the tile's keys;
//   online softmax in log2 units, the row maximum shared by the two lanes of
//     a row;
//   O^T += V^T P^T on the same MFMA: P^T (B operand) comes straight from the
//     lane's registers, split into a bf16 high part and the bf16 of the
//     remainder (two MFMAs, about 16 bits of the fp32 weight), and V^T (A
//     operand) is read from the value tile in LDS along the same key order.
// The chunk partials (running max, sum, unnormalized output) are combined in
// split order by a second kernel (deterministic).
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

// bf16 round-to-nearest-even of x and of the remainder x - bf16(x).
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
  hi = f32_to_bf16_rne(x);
  lo = f32_to_bf16_rne(x - bf16_to_f32(hi));
}

template <int D, int NQT>
__global__ __launch_bounds__(64 * NQT) void decode_kernel(
    Geo g, int32_t tq, int32_t nsplit, int32_t mp, const uint16_t* __restrict__ qn,
    int64_t q_sl, int64_t q_st, int64_t q_sh, const uint16_t* __restrict__ kp,
    const uint16_t* __restrict__ vp, const int64_t* __restrict__ poff,
    float* __restrict__ part_o, float2* __restrict__ part_ml) {
  constexpr int KS = D / 16;       // MFMA k-steps of S^T
  constexpr int HD = D / 2;        // dims per lane half in S^T
  constexpr int NDB = D / 32;      // 32-dim blocks of the output
  constexpr int RE = D + 8;        // padded LDS row, bf16 elements
  constexpr int CH = D / 8;        // 16-byte chunks per row
  constexpr int TILE_ELEMS = kDecTile * RE;
  __shared__ __align__(16) uint16_t lds[2][2][TILE_ELEMS];  // [buffer][K, V][row * RE]

  const int split = blockIdx.x;
  const int64_t u = blockIdx.y;
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
  const int M = tq * g.G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hh = lane >> 5;
  const int c32 = lane & 31;
  const int row = wave * 32 + c32;  // this lane's query row
  const float c2 = g.scale * kDecLog2e;

  // The query row as B fragments of S^T (zero for padding rows); lane half hh
  // owns the dims hh*HD .. hh*HD + HD - 1 (the contraction order is free).
  DecFrag qf[KS];
  {
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
  }

  // Cooperative tile staging: element e of the K and V tiles (row e / CH,
  // chunk e % CH); rows past the chunk end read as zero.
  constexpr int NTHR = 64 * NQT;
  constexpr int NCHUNKS = 2 * kDecTile * CH;
  constexpr int PER = (NCHUNKS + NTHR - 1) / NTHR;  // 16-byte chunks per thread
  uint4 stage[PER];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = threadIdx.x + j * NTHR;
      uint4 x = make_uint4(0u, 0u, 0u, 0u);
      if (e < NCHUNKS) {
        const int which = e / (kDecTile * CH);        // 0: K, 1: V
        const int r = (e / CH) % kDecTile, ch = e % CH;
        const int key = t0 + r;
        if (key < c1) {
          const uint16_t* src = (which ? vp : kp) + (p0 + key) * D + ch * 8;
          x = *reinterpret_cast<const uint4*>(src);
        }
      }
      stage[j] = x;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = threadIdx.x + j * NTHR;
      if (e < NCHUNKS) {
        const int which = e / (kDecTile * CH);
        const int r = (e / CH) % kDecTile, ch = e % CH;
        *reinterpret_cast<uint4*>(&lds[buf][which][r * RE + ch * 8]) = stage[j];
      }
    }
  };

  float m_run = -INFINITY, l_run = 0.f;
  dec_f32x16 O[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) O[db][v] = 0.f;

  load_tile(c0);
  store_tile(0);
  __syncthreads();
  for (int i = 0; i < ntiles; ++i) {
    const int t0 = c0 + i * kDecTile;
    const int buf = i & 1;
    if (i + 1 < ntiles) load_tile(t0 + kDecTile);
    const uint16_t* kt = lds[buf][0];
    const uint16_t* vt = lds[buf][1];
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
    // online softmax of the row (log2 units)
    float z[16];
    float mt = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = t0 + 8 * (v >> 2) + 4 * hh + (v & 3);
      z[v] = key < c1 ? s[v] * c2 : -INFINITY;
      mt = fmaxf(mt, z[v]);
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mnew = fmaxf(m_run, mt);
    const float alpha = __builtin_amdgcn_exp2f(m_run - mnew);
    m_run = mnew;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) O[db][v] *= alpha;
    // P^T fragments: k-step kk takes the lane's values v = 8 kk .. 8 kk + 7,
    // i.e. keys 16 kk + 8 (i/4) + 4 hh + i%4 for k-slot 8 hh + i
    DecFrag ph[2], pl[2];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float p = __builtin_amdgcn_exp2f(z[v] - mnew);
      l_run += p;
      split_bf16(p, ph[v >> 3].h[v & 7], pl[v >> 3].h[v & 7]);
    }
    // O^T += V^T P^T per 32-dim block; V^T lane (hh, c32) = dim 32 db + c32
    // over the same keys
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        DecFrag vf;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int key = 16 * kk + 8 * (i >> 2) + 4 * hh + (i & 3);
          vf.h[i] = vt[key * RE + 32 * db + c32];
        }
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, ph[kk].v, O[db], 0, 0, 0);
        O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pl[kk].v, O[db], 0, 0, 0);
      }
    }
    if (i + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // partials of this chunk: the row's (max, sum) and unnormalized output
  const float l_row = l_run + __shfl_xor(l_run, 32, 64);
  const int64_t pr = ((int64_t)u * nsplit + split) * mp + row;
  if (hh == 0) part_ml[pr] = make_float2(m_run, l_row);
  float* po = part_o + pr * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) po[32 * db + 8 * (v >> 2) + 4 * hh + (v & 3)] = O[db][v];
}

// Combine the chunk partials of each (unit, row) in split order.
template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(
    Geo g, int32_t tq, int32_t nsplit, int32_t mp, const int64_t* __restrict__ poff,
    const float* __restrict__ part_o, const float2* __restrict__ part_ml, float* __restrict__ out,
    float* __restrict__ lse) {
  const int64_t u = blockIdx.x;
  const int h = (int)(u % g.H);
  const int64_t lb = u / g.H;
  const int b = (int)(lb % g.B);
  const int l = (int)(lb / g.B);
  const int len = (int)(poff[u + 1] - poff[u]);
  const int nv = min(nsplit, (len + kDecKeys - 1) / kDecKeys);
  const int M = tq * g.G;
  const int Hq = g.H * g.G;
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int row = e / D, dd = e % D;
    float mx = -INFINITY;
    for (int sp = 0; sp < nv; ++sp) mx = fmaxf(mx, part_ml[((int64_t)u * nsplit + sp) * mp + row].x);
    float L = 0.f, acc = 0.f;
    for (int sp = 0; sp < nv; ++sp) {
      const int64_t pr = ((int64_t)u * nsplit + sp) * mp + row;
      const float2 ml = part_ml[pr];
      const float w = __builtin_amdgcn_exp2f(ml.x - mx);
      L += ml.y * w;
      acc += part_o[pr * D + dd] * w;
    }
    const int t = row / g.G, gq = row % g.G;
    const int64_t orow = ((int64_t)l * g.B * tq + (int64_t)b * tq + t) * Hq + h * g.G + gq;
    const float o = acc / L;
    if (!isfinite(o)) report_nonfinite(g);
    out[orow * D + dd] = o;
    if (lse && dd == 0) lse[orow] = (mx + __builtin_amdgcn_logf(L)) * kDecLn2;
  }
}

template <int D, int NQT>
static certkv_status launch_decode(const DecodeArgs& a, hipStream_t s) {
  const Geo& g = a.g;
  const int mp = NQT * 32;
  dim3 grid(a.nsplit, (unsigned)a.U);
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* kp = static_cast<const uint16_t*>(a.k_packed);
  const uint16_t* vp = static_cast<const uint16_t*>(a.v_packed);
  CERTKV_LAUNCH("decode", (decode_kernel<D, NQT>), grid, dim3(64 * NQT), 0, s, g, a.tq, a.nsplit,
                mp, q, a.q.s_layer, a.q.s_token, a.q.s_head, kp, vp, a.packed_offsets, a.part_o,
                a.part_ml);
  CERTKV_LAUNCH("decode_combine", decode_combine_kernel<D>, dim3((unsigned)a.U), dim3(256), 0, s,
                g, a.tq, a.nsplit, mp, a.packed_offsets, (const float*)a.part_o,
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
  return (size_t)U * nsplit * decode_nqt(tq * G) * 32;
}

int decode_nsplit(int max_len) { return (max_len + kDecKeys - 1) / kDecKeys; }

}  // namespace certkv
