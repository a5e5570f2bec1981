// Kept-key selection: threshold on the score order plus ballot compaction.
//
// The top-b keys of a unit (score descending, ties by position) are exactly
// the keys whose (radix key, position) pair is lexicographically <= the pair
// at rank b-1 of the sort.  One workgroup streams the unit's scores in
// position order (4096 positions per step, 4 consecutive per thread), tests
// each key against that threshold, and compacts the kept positions with wave
// ballots and a prefix over the 16 waves, so kept indices come out ascending
// without a scatter.  The same pass sums (s)_+ over the evicted
// keys and over all keys in fp64 (the tail mass and its normalizer).
#include "stages.h"

namespace certkv {

// budgets clamped to [0, n_b] (caller-supplied budgets in selection mode)
__global__ void clamp_budgets_kernel(Geo g, SeqTab st, int32_t* __restrict__ budgets) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int per_layer = st.count * g.H;
  if (i >= per_layer * g.L) return;
  const int l = i / per_layer, r = i % per_layer;
  const int bl = r / g.H, h = r % g.H;
  const int64_t u = unit_index(g, l, st.first + bl, h);
  int32_t b = budgets[u];
  b = b < 0 ? 0 : (b > st.len[bl] ? st.len[bl] : b);
  budgets[u] = b;
}

// Exclusive prefix over all units of the budgets -> kept_offsets[U+1];
// packed_offsets[u] = kept_offsets[u] + slot * u (slot = 1: one slot row per
// unit; 0 without the slot).
__global__ __launch_bounds__(1024) void offsets_kernel(int64_t U, int32_t slot,
                                                       const int32_t* __restrict__ budgets,
                                                       int64_t* __restrict__ kept_offsets,
                                                       int64_t* __restrict__ packed_offsets) {
  __shared__ int64_t wsum[16];
  __shared__ int64_t carry;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t base = 0; base < U; base += 1024) {
    const int64_t i = base + threadIdx.x;
    int64_t v = i < U ? (int64_t)budgets[i] : 0;
    int64_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      int64_t y = __shfl_up(incl, off, 64);
      if (lane >= off) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int64_t before = carry;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    if (i < U) {
      kept_offsets[i] = before + incl - v;
      if (packed_offsets) packed_offsets[i] = before + incl - v + slot * i;
    }
    __syncthreads();
    if (threadIdx.x == 1023) carry = before + incl;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    kept_offsets[U] = carry;
    if (packed_offsets) packed_offsets[U] = carry + slot * U;
  }
}

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelRounds = 8;                     // rounds of 1024 consecutive positions
constexpr int kSelTile = kSelThreads * kSelRounds; // 8192 positions per iteration
constexpr int kSelScanPer = kSelRounds * kSelWaves / 64;  // counts per lane of the scan

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    Geo g, SeqTab st, const float* __restrict__ scores, const uint32_t* __restrict__ sorted_keys,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ budgets,
    const int64_t* __restrict__ kept_offsets, int32_t* __restrict__ kept_idx, int64_t capacity,
    double* __restrict__ evicted_sum, double* __restrict__ total_sum, uint64_t* __restrict__ bm,
    int32_t bm_stride) {
  // kept counts of each (round, wave) of a tile, then their exclusive prefix
  // in position order (round-major); the tile's total at the end
  __shared__ uint32_t kcnt[kSelRounds * kSelWaves + 1];
  __shared__ double dsum[2][kSelWaves];
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t base = lht_base(g, l, h, st.start[bl]);
  const int64_t u = unit_index(g, l, b, h);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int bb = budgets[u];
  const int wkeep = n - g.keep_w;  // first kept-window position (n: none)
  uint32_t kthr = 0u;
  int32_t ithr = -1;  // keep nothing when bb == 0
  if (bb > 0 && bb <= n) {
    kthr = sorted_keys[base + bb - 1];
    ithr = perm[base + bb - 1];
  }
  const int64_t off = kept_offsets[u];
  int64_t run = 0;
  double se = 0.0, sa = 0.0;
  // Round r of a tile: positions j0 + 1024 r + thread, so every load covers
  // 256 consecutive bytes per wave.  Loads through a range-checked buffer:
  // positions past the end read as zero, so no branch sits around them and
  // the next tile's loads stay in flight while this one is tested; they are
  // masked where used.
  const BufRsrc srs = make_rsrc(scores + base, (uint32_t)n * 4u);
  auto load = [&](int j0, float (&sv)[kSelRounds]) {
#pragma unroll
    for (int r = 0; r < kSelRounds; ++r)
      sv[r] = __uint_as_float(
          buf_load_u32(srs, (uint32_t)(j0 + r * kSelThreads + (int)threadIdx.x) * 4u));
  };
  float cur[kSelRounds], nxt[kSelRounds];
  load(0, cur);
  for (int j0 = 0; j0 < n; j0 += kSelTile) {
    load(j0 + kSelTile, nxt);
    uint32_t kmask = 0;
    uint64_t bal[kSelRounds];  // wave-uniform: scalar registers
#pragma unroll
    for (int r = 0; r < kSelRounds; ++r) {
      const int j = j0 + r * kSelThreads + (int)threadIdx.x;
      const bool valid = j < n;
      const uint32_t key = desc_key(cur[r]);
      // kept window keys hold ranks 0..w-1 in position order; the others
      // are kept up to the threshold pair at rank bb-1
      const bool keep = valid && (j >= wkeep ? (j - wkeep < bb)
                                             : (bb > g.keep_w && (key < kthr || (key == kthr && j <= ithr))));
      const double sp = (valid && cur[r] > 0.f) ? (double)cur[r] : 0.0;
      sa += sp;
      se += keep ? 0.0 : sp;
      bal[r] = __ballot(keep);
      kmask |= (uint32_t)keep << r;
      if (lane == 0) {
        kcnt[r * kSelWaves + wave] = (uint32_t)__popcll(bal[r]);
        // kept bitmap: the ballot is the word of the wave's 64 positions
        const int widx = ((j0 + r * kSelThreads) >> 6) + wave;
        if (bm && widx < bm_stride) bm[u * bm_stride + widx] = bal[r];
      }
    }
    __syncthreads();
    // exclusive prefix of the counts in position order (one wave)
    if (wave == 0) {
      uint32_t c[kSelScanPer], t = 0;
#pragma unroll
      for (int i = 0; i < kSelScanPer; ++i) {
        c[i] = kcnt[kSelScanPer * lane + i];
        t += c[i];
      }
      uint32_t incl = t;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      uint32_t ex = incl - t;
#pragma unroll
      for (int i = 0; i < kSelScanPer; ++i) {
        kcnt[kSelScanPer * lane + i] = ex;
        ex += c[i];
      }
      if (lane == 63) kcnt[kSelRounds * kSelWaves] = incl;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSelRounds; ++r) {
      if ((kmask >> r) & 1u) {
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(bal[r] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal[r], 0u));
        const int64_t dst = off + run + kcnt[r * kSelWaves + wave] + below;
        if (dst < capacity) kept_idx[dst] = j0 + r * kSelThreads + (int)threadIdx.x;
      }
    }
    run += kcnt[kSelRounds * kSelWaves];
#pragma unroll
    for (int r = 0; r < kSelRounds; ++r) cur[r] = nxt[r];
  }
  se = wave_sum(se);
  sa = wave_sum(sa);
  if (lane == 0) {
    dsum[0][wave] = se;
    dsum[1][wave] = sa;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double e = 0.0, t = 0.0;
    for (int w = 0; w < kSelWaves; ++w) {
      e += dsum[0][w];
      t += dsum[1][w];
    }
    if (evicted_sum) evicted_sum[u] = e;
    if (total_sum) total_sum[u] = t;
  }
}

// Coverage budget k_eta: the normalizer sum (s)_+ in position order, then the
// rank-order prefix of a = (s)_+ / sum until it reaches retain, both summed
// one term at a time in fp64 (one wave per unit, uniform accumulators).
__global__ __launch_bounds__(64) void coverage_kernel(Geo g, SeqTab st, const float* __restrict__ scores,
                                                      const uint32_t* __restrict__ sorted_keys,
                                                      double retain, int32_t* __restrict__ budgets) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int b = st.first + bl;
  const int n = st.len[bl];
  const int64_t base = lht_base(g, l, h, st.start[bl]);
  const int lane = threadIdx.x;
  double tot = 0.0;
  for (int j0 = 0; j0 < n; j0 += 64) {
    const int j = j0 + lane;
    const float s = j < n ? scores[base + j] : 0.f;
    const double sp = s > 0.f ? (double)s : 0.0;
    const int cnt = min(64, n - j0);
    for (int i = 0; i < cnt; ++i) tot += __shfl(sp, i, 64);
  }
  const double inv_n = 1.0 / (double)n;
  double p = 0.0;
  int k = n;
  bool done = false;
  for (int r0 = 0; r0 < n && !done; r0 += 64) {
    const int r = r0 + lane;
    const float s = r < n ? desc_key_value(sorted_keys[base + r]) : 0.f;
    const double a = tot > 0.0 ? (s > 0.f ? (double)s / tot : 0.0) : inv_n;
    const int cnt = min(64, n - r0);
    for (int i = 0; i < cnt; ++i) {
      p += __shfl(a, i, 64);
      if (p >= retain) {
        k = r0 + i + 1;
        done = true;
        break;
      }
    }
  }
  // a kept window leads the order and is never cut
  if (g.keep_w) k = max(k, min(g.keep_w, n));
  if (lane == 0) budgets[unit_index(g, l, b, h)] = k;
}


certkv_status run_coverage(const Geo& g, const SeqTab& st, const float* scores,
                           const uint32_t* sorted_keys, double retain, int32_t* budgets,
                           hipStream_t s) {
  CERTKV_LAUNCH("coverage_budget", coverage_kernel, dim3(g.H * st.count, g.L), dim3(64), 0, s, g, st,
                scores, sorted_keys, retain, budgets);
  return CERTKV_OK;
}

certkv_status run_clamp(const Geo& g, const SeqTab& st, int32_t* budgets, hipStream_t s) {
  const int total = st.count * g.H * g.L;
  CERTKV_LAUNCH("clamp_budgets", clamp_budgets_kernel, dim3((total + 255) / 256), dim3(256), 0, s, g,
                st, budgets);
  return CERTKV_OK;
}

certkv_status run_offsets(int64_t U, int32_t slot, const int32_t* budgets, int64_t* kept_offsets,
                          int64_t* packed_offsets, hipStream_t s) {
  CERTKV_LAUNCH("kept_offsets", offsets_kernel, dim3(1), dim3(1024), 0, s, U, slot, budgets,
                kept_offsets, packed_offsets);
  return CERTKV_OK;
}

__global__ void packed_from_kept_kernel(int64_t U, int32_t slot,
                                        const int64_t* __restrict__ kept_offsets,
                                        int64_t* __restrict__ packed_offsets) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= U) packed_offsets[i] = kept_offsets[i] + slot * i;
}

certkv_status run_packed_from_kept(int64_t U, int32_t slot, const int64_t* kept_offsets,
                                   int64_t* packed_offsets, hipStream_t s) {
  CERTKV_LAUNCH("packed_offsets", packed_from_kept_kernel, dim3((unsigned)((U + 256) / 256)),
                dim3(256), 0, s, U, slot, kept_offsets, packed_offsets);
  return CERTKV_OK;
}

// True-uniform allocation (one-factor ablation): every head of a (layer,
// sequence) gets B_real / H, which the budget algebra makes whole.
__global__ void uniform_budgets_kernel(Geo g, SeqTab st, int32_t* __restrict__ budgets) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int total = st.count * g.H * g.L;
  if (i >= total) return;
  const int h = i % g.H;
  const int bi = (i / g.H) % st.count;
  const int l = i / (g.H * st.count);
  budgets[unit_index(g, l, st.first + bi, h)] = (int32_t)(st.b_real[bi] / g.H);
}

certkv_status run_uniform_budgets(const Geo& g, const SeqTab& st, int32_t* budgets, hipStream_t s) {
  const int total = st.count * g.H * g.L;
  CERTKV_LAUNCH("uniform_budgets", uniform_budgets_kernel, dim3((total + 255) / 256), dim3(256), 0,
                s, g, st, budgets);
  return CERTKV_OK;
}

// Kept mask [L][H][T] uint8: cleared with 16-byte stores (the mask base is
// 16-byte aligned; the tail of the buffer byte by byte), then the kept
// positions of every unit set to 1.
__global__ __launch_bounds__(256) void mask_clear_kernel(uint8_t* __restrict__ mask, int64_t bytes) {
  const int64_t nvec = bytes / 16;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride)
    reinterpret_cast<uint4*>(mask)[i] = make_uint4(0u, 0u, 0u, 0u);
  if (blockIdx.x == 0)
    for (int64_t i = nvec * 16 + threadIdx.x; i < bytes; i += blockDim.x) mask[i] = 0;
}

__global__ __launch_bounds__(256) void mask_set_kernel(Geo g, SeqTab st,
                                                        const int64_t* __restrict__ kept_offsets,
                                                        const int32_t* __restrict__ kept_idx,
                                                        uint8_t* __restrict__ mask) {
  const int h = blockIdx.x % g.H;
  const int bl = blockIdx.x / g.H;
  const int l = blockIdx.y;
  if (bl >= st.count) return;
  const int n = st.len[bl];
  const int64_t u = unit_index(g, l, st.first + bl, h);
  const int64_t base = lht_base(g, l, h, st.start[bl]);
  const int64_t k0 = kept_offsets[u], k1 = kept_offsets[u + 1];
  for (int64_t i = k0 + threadIdx.x; i < k1; i += blockDim.x) {
    const int j = kept_idx[i];
    if (j >= 0 && j < n) mask[base + j] = 1;
  }
}

certkv_status run_mask(const Geo& g, const std::vector<SeqTab>& tabs, const int64_t* kept_offsets,
                       const int32_t* kept_idx, uint8_t* mask, hipStream_t s) {
  const int64_t bytes = (int64_t)g.L * g.H * g.T;
  const int64_t nvec = bytes / 16;
  const unsigned blocks = (unsigned)(nvec / 256 + 1 < 4096 ? nvec / 256 + 1 : 4096);
  CERTKV_LAUNCH("kept_mask_clear", mask_clear_kernel, dim3(blocks), dim3(256), 0, s, mask, bytes);
  for (const SeqTab& t : tabs)
    CERTKV_LAUNCH("kept_mask_set", mask_set_kernel, dim3(g.H * t.count, g.L), dim3(256), 0, s, g, t,
                  kept_offsets, kept_idx, mask);
  return CERTKV_OK;
}

certkv_status run_select(const SelectArgs& a, const SeqTab& st, hipStream_t s) {
  CERTKV_LAUNCH("select", select_kernel, dim3(a.g.H * st.count, a.g.L), dim3(kSelThreads), 0, s, a.g, st,
                a.scores, a.sorted_keys, a.perm, (const int32_t*)a.budgets,
                (const int64_t*)a.kept_offsets, a.kept_idx, a.capacity, a.evicted_sum, a.total_sum,
                a.bitmap, a.bm_stride);
  return CERTKV_OK;
}

}  // namespace certkv
