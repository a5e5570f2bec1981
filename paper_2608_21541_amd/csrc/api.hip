// C ABI of libcertkv.so: argument validation, workspace layout, launch order.
#include <math.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "stages.h"

namespace certkv {

// ---- profiling -------------------------------------------------------------
namespace {
struct ProfRec {
  std::string name;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_pool;

hipEvent_t pool_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

void prof_begin(const char* name, hipStream_t s) {
  if (!g_prof_on) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfRec r{name, pool_event(), pool_event()};
  if (r.a) hipEventRecord(r.a, s);
  g_prof.push_back(r);
}

void prof_end(hipStream_t s) {
  if (!g_prof_on) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof.empty() && g_prof.back().b) hipEventRecord(g_prof.back().b, s);
}

// ---- problem description ----------------------------------------------------
struct Plan {
  Geo g;
  int32_t dtype;
  int64_t U;         // units
  int max_len;
  int M;             // window rows per unit
  int kpb;           // keys per scoring block, pass 1
  int nkb_max;       // pass-1 scoring blocks per unit (max over sequences)
  int kpb2;          // keys per scoring block, pass 2
  int nkb2_max;      // pass-2 scoring blocks per unit
  int nblk_max;      // 256-rank allocation blocks per unit
  int nsub_max;      // 16-rank allocation sub-blocks per unit
  int bm_words;      // 64-bit bitmap words per unit
  int nsplit;        // tail gather workgroups per unit
  int alloc;         // allocator: 0 Lagrangian + repair, 1 uniform, 2 greedy marginal
  const int64_t* cu;
};

static certkv_status make_plan(const certkv_problem* p, Plan* pl) {
  if (!p) return CERTKV_EINVAL;
  if (p->num_layers < 1 || p->batch < 1 || p->num_kv_heads < 1 || p->group < 1 || p->window < 1)
    return CERTKV_EINVAL;
  if (p->num_kv_heads > 64) return CERTKV_EUNSUPPORTED;
  if (p->head_dim != 64 && p->head_dim != 128) return CERTKV_EUNSUPPORTED;
  if (!p->cu_seqlens_host) return CERTKV_EINVAL;
  if (p->q_dtype != p->kv_dtype) return CERTKV_EUNSUPPORTED;
  if (p->kv_dtype != CERTKV_F32 && p->kv_dtype != CERTKV_BF16) return CERTKV_EUNSUPPORTED;
  if (p->flags & ~(uint32_t)(CERTKV_CAUSAL | CERTKV_DRY_RUN | CERTKV_KEEP_WINDOW |
                             CERTKV_STAT_UNCENTERED | CERTKV_STAT_TAIL_MASS |
                             CERTKV_ALLOC_UNIFORM | CERTKV_ALLOC_GREEDY | CERTKV_NO_SLOT))
    return CERTKV_EINVAL;
  if ((p->flags & CERTKV_STAT_UNCENTERED) && (p->flags & CERTKV_STAT_TAIL_MASS))
    return CERTKV_EINVAL;
  if ((p->flags & CERTKV_ALLOC_UNIFORM) && (p->flags & CERTKV_ALLOC_GREEDY))
    return CERTKV_EINVAL;
  if (!(p->softmax_scale >= 0.f) || isinf(p->softmax_scale)) return CERTKV_EINVAL;
  const int64_t* cu = p->cu_seqlens_host;
  if (cu[0] != 0) return CERTKV_EINVAL;
  int max_len = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int64_t nb = cu[b + 1] - cu[b];
    if (nb < p->window || nb > (int64_t)0x7fffffff - 1024) return CERTKV_EINVAL;
    if (nb > max_len) max_len = (int)nb;
  }
  const int M = p->window * p->group;
  if (p->q_dtype == CERTKV_BF16 && M > 512) return CERTKV_EUNSUPPORTED;
  if (p->q_dtype == CERTKV_F32 && (int64_t)M * p->head_dim > 16384) return CERTKV_EUNSUPPORTED;
  Plan& P = *pl;
  P.g.L = p->num_layers;
  P.g.B = p->batch;
  P.g.H = p->num_kv_heads;
  P.g.G = p->group;
  P.g.D = p->head_dim;
  P.g.w = p->window;
  P.g.T = cu[p->batch];
  P.g.scale = p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / sqrtf((float)p->head_dim);
  P.g.causal = (p->flags & CERTKV_CAUSAL) ? 1 : 0;
  P.g.status = p->dev_status;
  P.g.keep_w = (p->flags & CERTKV_KEEP_WINDOW) ? p->window : 0;
  P.g.stat = (p->flags & CERTKV_STAT_UNCENTERED) ? 1 : (p->flags & CERTKV_STAT_TAIL_MASS) ? 2 : 0;
  P.g.slot = (p->flags & CERTKV_NO_SLOT) ? 0 : 1;
  P.alloc = (p->flags & CERTKV_ALLOC_UNIFORM) ? 1 : (p->flags & CERTKV_ALLOC_GREEDY) ? 2 : 0;
  P.dtype = p->kv_dtype;
  P.U = (int64_t)P.g.L * P.g.B * P.g.H;
  P.max_len = max_len;
  P.M = M;
  P.cu = cu;
  // Scoring blocks: as long as the grid keeps about four workgroups per
  // resident slot (pass 1 holds two 8-wave workgroups per CU, pass 2 with
  // its key-sum registers one), larger blocks amortize the staging of the
  // window queries and the per-block reduction.
  int kpb = 256, kpb2 = 256;
  if (P.dtype == CERTKV_BF16) {
    constexpr int64_t kCUs = 256;
    auto grow = [&](int64_t min_wgs) {
      int k = 512;
      while (k < 65536 && P.U * ((max_len + 2 * k - 1) / (2 * k)) >= min_wgs) k *= 2;
      return k;
    };
    kpb = grow(4 * 2 * kCUs);
    kpb2 = grow(4 * kCUs);
  }
  P.kpb = kpb;
  P.nkb_max = (max_len + kpb - 1) / kpb;
  P.kpb2 = kpb2;
  P.nkb2_max = (max_len + kpb2 - 1) / kpb2;
  P.nblk_max = (max_len + 255) / 256;
  P.nsub_max = (max_len + 15) / 16;
  P.bm_words = (max_len + 63) / 64;
  // tail gather: one workgroup per 2048 positions of the longest sequence
  // (about 200 kept rows each at a tenth kept), at most 128 per unit
  P.nsplit = (max_len + 2047) / 2048;
  if (P.nsplit > 128) P.nsplit = 128;
  return CERTKV_OK;
}

static certkv_status check_tensor(const certkv_tensor& t, const Plan& P) {
  if (!t.ptr) return CERTKV_EINVAL;
  if (((uintptr_t)t.ptr & 15u) != 0) return CERTKV_EINVAL;
  if ((t.s_layer % 8) || (t.s_token % 8) || (t.s_head % 8)) return CERTKV_EINVAL;
  if (t.s_layer < 0 || t.s_token < 0 || t.s_head < 0) return CERTKV_EINVAL;
  // the rows of one (layer, head, sequence) are addressed with 32-bit byte
  // offsets from the slice start
  const int64_t esz = P.dtype == CERTKV_BF16 ? 2 : 4;
  if (((int64_t)(P.max_len - 1) * t.s_token + P.g.D) * esz > (int64_t)0xFFFFFFFFLL)
    return CERTKV_EUNSUPPORTED;
  return CERTKV_OK;
}

// Sequence tables of at most kMaxSeq sequences each.
static std::vector<SeqTab> make_tabs(const Plan& P, const int32_t* n_keep, double alpha) {
  std::vector<SeqTab> out;
  for (int b0 = 0; b0 < P.g.B; b0 += kMaxSeq) {
    SeqTab t;
    memset(&t, 0, sizeof(t));
    t.first = b0;
    t.count = P.g.B - b0 < kMaxSeq ? P.g.B - b0 : kMaxSeq;
    for (int i = 0; i < t.count; ++i) {
      const int b = b0 + i;
      t.start[i] = P.cu[b];
      t.len[i] = (int32_t)(P.cu[b + 1] - P.cu[b]);
      if (n_keep) {
        t.n_keep[i] = n_keep[b];
        const int64_t br = (int64_t)P.g.H * n_keep[b] - (P.g.slot ? P.g.H : 0);
        int64_t bm = (int64_t)floor(alpha * (double)br / (double)P.g.H);
        if (bm < 1) bm = 1;
        t.b_real[i] = br;
        t.b_min[i] = (int32_t)bm;
      }
    }
    out.push_back(t);
  }
  return out;
}

static certkv_status check_budget(const Plan& P, const int32_t* n_keep, double alpha, int steps) {
  if (!n_keep) return CERTKV_EINVAL;
  if (!(alpha >= 0.f && alpha <= 1.f)) return CERTKV_EINVAL;
  if (steps < 0 || steps > 200) return CERTKV_EINVAL;
  for (int b = 0; b < P.g.B; ++b) {
    const int64_t nb = P.cu[b + 1] - P.cu[b];
    // with the slot 2 <= n_keep <= n; without it every live row is a real
    // key and a head keeps at most n - 1 of them
    if (P.g.slot ? (n_keep[b] < 2 || n_keep[b] > nb) : (n_keep[b] < 1 || n_keep[b] > nb - 1))
      return CERTKV_EINFEASIBLE;
    const int64_t br = (int64_t)P.g.H * n_keep[b] - (P.g.slot ? P.g.H : 0);
    int64_t bm = (int64_t)floor(alpha * (double)br / (double)P.g.H);
    if (bm < 1) bm = 1;
    if (bm > nb - 1 || (int64_t)P.g.H * bm > br) return CERTKV_EINFEASIBLE;
    if (P.g.keep_w && bm < P.g.keep_w) return CERTKV_EINFEASIBLE;
  }
  return CERTKV_OK;
}

// ---- workspace layout ------------------------------------------------------
struct WS {
  size_t off = 0;
  char* base = nullptr;
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

struct Bufs {
  // scoring
  float2* part = nullptr;
  float* lse2 = nullptr;
  float* kpart = nullptr;
  int32_t* flag = nullptr;
  double* ksum = nullptr;
  // order / curves / allocation
  uint32_t *keysA = nullptr, *keysB = nullptr;
  int32_t *valsA = nullptr, *valsB = nullptr;
  int32_t* perm = nullptr;
  double* ssum = nullptr;
  float* curves = nullptr;
  float* cmin = nullptr;
  float* cmaxb = nullptr;
  int32_t* cpos = nullptr;
  double* dmax = nullptr;
  double* vsum = nullptr;
  int64_t* repairs = nullptr;
  int32_t* alloc_sync = nullptr;
  // select / tail
  uint64_t* bitmap = nullptr;
  int64_t* kept_offsets = nullptr;
  double* tpart = nullptr;
  double* mpart = nullptr;
  double* evicted_sum = nullptr;
  double* total_sum = nullptr;
};

enum : uint32_t {
  NEED_SCORE = 1u,
  NEED_SORT = 2u,
  NEED_CURVES = 4u,
  NEED_MINMAX = 8u,
  NEED_BITMAP = 16u,
  NEED_KSUM = 32u,
  NEED_PERM = 64u,
  NEED_CURVEBUF = 128u,
  NEED_OFFSETS = 256u,
};

static size_t layout(const Plan& P, uint32_t need, void* ws, Bufs* b) {
  WS w;
  w.base = static_cast<char*>(ws);
  const size_t LHT = (size_t)P.g.L * P.g.H * (size_t)P.g.T;
  if (need & NEED_SCORE) {
    b->part = w.take<float2>((size_t)P.U * P.nkb_max * P.M);
    b->lse2 = w.take<float>((size_t)P.U * P.M);
    b->kpart = w.take<float>((size_t)P.U * P.nkb2_max * P.g.D);
    b->flag = w.take<int32_t>((size_t)P.U);
  }
  if (need & NEED_KSUM) {
    b->ksum = w.take<double>((size_t)P.U * P.g.D);
    b->vsum = w.take<double>((size_t)P.U * P.g.D);
  }
  if (need & NEED_SORT) {
    b->keysA = w.take<uint32_t>(LHT);
    b->keysB = w.take<uint32_t>(LHT);
    b->valsA = w.take<int32_t>(LHT);
    b->valsB = w.take<int32_t>(LHT);
    b->ssum = w.take<double>((size_t)P.U);
  }
  if (need & NEED_PERM) b->perm = w.take<int32_t>(LHT);
  if (need & NEED_CURVEBUF) b->curves = w.take<float>(LHT);
  if (need & (NEED_CURVES | NEED_MINMAX)) {
    b->cmin = w.take<float>((size_t)P.U * P.nblk_max * 2);
    b->cmaxb = w.take<float>((size_t)P.U * P.nblk_max);
    b->cpos = w.take<int32_t>((size_t)P.U * P.nblk_max);
    b->dmax = w.take<double>((size_t)P.U * P.nblk_max);
    b->repairs = w.take<int64_t>((size_t)P.g.L * P.g.B * 3);
    b->alloc_sync = w.take<int32_t>(alloc_sync_words());
  }
  if (need & NEED_BITMAP) {
    b->bitmap = w.take<uint64_t>((size_t)P.U * P.bm_words);
    b->tpart = w.take<double>((size_t)P.U * P.nsplit * 2 * P.g.D);
    b->mpart = w.take<double>((size_t)P.U * P.nsplit * 3);
    b->evicted_sum = w.take<double>((size_t)P.U);
    b->total_sum = w.take<double>((size_t)P.U);
  }
  if (need & NEED_OFFSETS) b->kept_offsets = w.take<int64_t>((size_t)P.U + 1);
  return (w.off + 255) & ~(size_t)255;
}

static uint32_t stage_needs(int32_t stage) {
  switch (stage) {
    case CERTKV_STAGE_SCORE:
      return NEED_SCORE;
    case CERTKV_STAGE_ALLOCATE:
      return NEED_SORT | NEED_CURVES | NEED_PERM | NEED_CURVEBUF;
    case CERTKV_STAGE_SELECT:
      return NEED_SORT | NEED_PERM;
    case CERTKV_STAGE_TAIL:
      return NEED_BITMAP;
    case CERTKV_STAGE_COMPACT:
      return 0;
    case CERTKV_STAGE_COMPRESS:
      return NEED_SCORE | NEED_KSUM | NEED_SORT | NEED_CURVES | NEED_PERM | NEED_CURVEBUF |
             NEED_BITMAP;
    default:
      return 0xffffffffu;
  }
}

static certkv_status check_ws(const Plan& P, uint32_t need, void* ws, size_t bytes, Bufs* b) {
  const size_t req = layout(P, need, nullptr, b);
  if (req > 0) {
    if (!ws) return CERTKV_EWORKSPACE;
    if (((uintptr_t)ws & 255u) != 0) return CERTKV_EINVAL;
    if (bytes < req) return CERTKV_EWORKSPACE;
  }
  *b = Bufs();
  layout(P, need, ws, b);
  return CERTKV_OK;
}

#define TRY(x)                         \
  do {                                 \
    certkv_status _s = (x);            \
    if (_s != CERTKV_OK) return _s;    \
  } while (0)

// ---- stage drivers -----------------------------------------------------------
static certkv_status do_score(const Plan& P, certkv_tensor q, certkv_tensor k,
                              const float* lse_in, float* scores, double* ksum, float* lse_out,
                              const Bufs& w, hipStream_t s) {
  ScoreArgs a;
  a.g = P.g;
  a.lse_in = lse_in;
  a.lse_out = lse_out;
  a.q = q;
  a.k = k;
  a.dtype = P.dtype;
  a.scores = scores;
  a.ksum = ksum;
  a.part = w.part;
  a.lse2 = w.lse2;
  a.kpart = w.kpart;
  a.flag = w.flag;
  a.keys_per_block = P.dtype == CERTKV_BF16 ? P.kpb : 256;
  a.nkb_max = P.dtype == CERTKV_BF16 ? P.nkb_max : (P.max_len + 255) / 256;
  a.keys_per_block2 = P.dtype == CERTKV_BF16 ? P.kpb2 : 256;
  a.nkb2_max = P.dtype == CERTKV_BF16 ? P.nkb2_max : (P.max_len + 255) / 256;
  for (const SeqTab& t : make_tabs(P, nullptr, 0.f)) {
    int ml = 0;
    for (int i = 0; i < t.count; ++i) ml = t.len[i] > ml ? t.len[i] : ml;
    TRY(run_score(a, t, ml, s));
  }
  return CERTKV_OK;
}

static certkv_status do_sort(const Plan& P, const float* scores, int32_t* perm, const Bufs& w,
                             hipStream_t s) {
  SortArgs a;
  a.g = P.g;
  a.scores = scores;
  a.keysA = w.keysA;
  a.keysB = w.keysB;
  a.keys_out = w.keysA;
  a.valsA = w.valsA;
  a.valsB = w.valsB;
  a.perm_out = perm;
  a.ssum = w.ssum;
  for (const SeqTab& t : make_tabs(P, nullptr, 0.f)) TRY(run_sort(a, t, s));
  return CERTKV_OK;
}

static certkv_status do_curves(const Plan& P, certkv_tensor v, const int32_t* perm, float* curves,
                               double* vsum, const Bufs& w, hipStream_t s) {
  CurveArgs a;
  a.g = P.g;
  a.sorted_keys = w.keysA;
  a.perm = perm;
  a.ssum = w.ssum;
  a.v = v;
  a.dtype = P.dtype;
  a.curves = curves;
  a.vsum = vsum;
  for (const SeqTab& t : make_tabs(P, nullptr, 0.f)) TRY(run_curves(a, t, s));
  return CERTKV_OK;
}

static certkv_status do_allocate(const Plan& P, const float* curves, const int32_t* n_keep,
                                 double alpha, int steps, int32_t* budgets, bool minmax,
                                 const Bufs& w, hipStream_t s, int64_t* stats = nullptr) {
  AllocArgs a;
  a.g = P.g;
  a.curves = curves;
  a.cmin = w.cmin;
  a.cmaxb = w.cmaxb;
  a.cpos = w.cpos;
  a.dmax = w.dmax;
  a.nblk_max = P.nblk_max;
  a.steps = P.alloc == 2 ? 0 : steps;  // greedy marginal: the repair from b_min
  a.budgets = budgets;
  a.repairs = stats ? stats : w.repairs;
  a.sync = w.alloc_sync;
  (void)minmax;
  for (const SeqTab& t : make_tabs(P, n_keep, alpha)) {
    if (P.alloc == 1)
      TRY(run_uniform_budgets(P.g, t, budgets, s));
    else
      TRY(run_allocate(a, t, s));
  }
  return CERTKV_OK;
}

static certkv_status do_select(const Plan& P, const float* scores, const uint32_t* sorted_keys,
                               const int32_t* perm, int32_t* budgets, int mode, double retain,
                               int64_t* kept_offsets, int64_t* packed_offsets, int32_t* kept_idx,
                               int64_t capacity, const Bufs* fused, hipStream_t s) {
  const auto tabs = make_tabs(P, nullptr, 0.f);
  for (const SeqTab& t : tabs) {
    if (mode == CERTKV_SELECT_COVERAGE)
      TRY(run_coverage(P.g, t, scores, sorted_keys, retain, budgets, s));
    else if (!fused)  // the pass's own budgets lie in [b_min, n - 1] already
      TRY(run_clamp(P.g, t, budgets, s));
  }
  TRY(run_offsets(P.U, P.g.slot, budgets, kept_offsets, packed_offsets, s));
  SelectArgs a;
  a.g = P.g;
  a.scores = scores;
  a.sorted_keys = sorted_keys;
  a.perm = perm;
  a.budgets = budgets;
  a.kept_offsets = kept_offsets;
  a.packed_offsets = packed_offsets;
  a.kept_idx = kept_idx;
  a.capacity = capacity;
  a.evicted_sum = fused ? fused->evicted_sum : nullptr;
  a.total_sum = fused ? fused->total_sum : nullptr;
  a.bitmap = fused ? fused->bitmap : nullptr;
  a.bm_stride = P.bm_words;
  for (const SeqTab& t : tabs) TRY(run_select(a, t, s));
  return CERTKV_OK;
}

static certkv_status do_tail(const Plan& P, const float* scores, certkv_tensor k, certkv_tensor v,
                             const int64_t* kept_offsets, const int32_t* kept_idx,
                             const double* ksum, const double* vsum, float* k_star, float* v_star,
                             double* tail_mass, void* k_packed, void* v_packed,
                             int32_t* pos_packed, bool do_tail, bool do_compact, bool fused,
                             const Bufs& w, hipStream_t s) {
  TailArgs a;
  a.g = P.g;
  a.dtype = P.dtype;
  a.scores = scores;
  a.k = k;
  a.v = v;
  a.kept_offsets = kept_offsets;
  a.kept_idx = kept_idx;
  a.bitmap = w.bitmap;
  a.bm_stride = P.bm_words;
  a.nsplit = P.nsplit;
  a.kpart = w.tpart;
  a.mpart = w.mpart;
  a.evicted_sum = fused ? w.evicted_sum : nullptr;
  a.total_sum = fused ? w.total_sum : nullptr;
  a.ksum = ksum;
  a.vsum = vsum;
  a.k_star = k_star;
  a.v_star = v_star;
  a.tail_mass = tail_mass;
  a.k_packed = k_packed;
  a.v_packed = v_packed;
  a.pos_packed = pos_packed;
  a.do_tail = do_tail;
  a.do_compact = do_compact;
  const auto tabs = make_tabs(P, nullptr, 0.f);
  if (do_tail && !fused) {
    bool first = true;
    for (const SeqTab& t : tabs) {
      TRY(run_bitmap(a, t, P.U * (int64_t)P.bm_words, first, s));
      first = false;
    }
  }
  for (const SeqTab& t : tabs) TRY(run_tail(a, t, s));
  return CERTKV_OK;
}

}  // namespace certkv

using namespace certkv;

extern "C" {

const char* certkv_status_string(certkv_status st) {
  switch (st) {
    case CERTKV_OK:
      return "ok";
    case CERTKV_EINVAL:
      return "invalid argument";
    case CERTKV_EUNSUPPORTED:
      return "unsupported configuration";
    case CERTKV_EINFEASIBLE:
      return "infeasible budget (need 2 <= n_keep <= n, and b_min >= w with a kept window)";
    case CERTKV_ENONFINITE:
      return "non-finite input";
    case CERTKV_EWORKSPACE:
      return "workspace too small";
    case CERTKV_EHIP:
      return "HIP runtime error";
    case CERTKV_ERANGE:
      return "packed segment longer than the decode row bound";
    default:
      return "unknown status";
  }
}

size_t certkv_workspace_size(const certkv_problem* p, int32_t stage) {
  Plan P;
  if (make_plan(p, &P) != CERTKV_OK) return 0;
  const uint32_t need = stage_needs(stage);
  if (need == 0xffffffffu) return 0;
  Bufs b;
  return layout(P, need, nullptr, &b);
}

certkv_status certkv_score(const certkv_problem* p, certkv_tensor q_win, certkv_tensor k,
                           const float* lse_in, float* scores, double* ksum, float* lse_out,
                           void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(q_win, P));
  TRY(check_tensor(k, P));
  if (!scores) return CERTKV_EINVAL;
  Bufs w;
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_SCORE), ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  return do_score(P, q_win, k, lse_in, scores, ksum, lse_out, w, (hipStream_t)stream);
}

}  // extern "C"

// ---- scoring without a caller workspace ---------------------------------------
// The workspace of certkv_score_noalloc: a fixed device array (every device
// the library runs on holds its own copy until the process ends).  Host code
// never uses the symbol itself as an address: the device address is looked
// up once per device with hipGetSymbolAddress, with that device current.
namespace certkv {
namespace {
constexpr size_t kScratchBytes = (size_t)64 << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

static certkv_status scratch_base(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CERTKV_EHIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return CERTKV_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CERTKV_OK;
}
}  // namespace certkv

extern "C" {

size_t certkv_score_noalloc_max_bytes(void) { return kScratchBytes; }

certkv_status certkv_score_noalloc(const certkv_problem* p, certkv_tensor q_win,
                                   certkv_tensor k, const float* lse_in, float* scores,
                                   double* ksum, float* lse_out, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(q_win, P));
  TRY(check_tensor(k, P));
  if (!scores) return CERTKV_EINVAL;
  Bufs w;
  const size_t need = layout(P, stage_needs(CERTKV_STAGE_SCORE), nullptr, &w);
  if (need > kScratchBytes) return CERTKV_EWORKSPACE;
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  void* ws = nullptr;
  TRY(scratch_base(&ws));
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_SCORE), ws, kScratchBytes, &w));
  return do_score(P, q_win, k, lse_in, scores, ksum, lse_out, w, (hipStream_t)stream);
}

certkv_status certkv_allocate(const certkv_problem* p, const float* scores, certkv_tensor v,
                              const int32_t* n_keep_host, double alpha, int32_t steps,
                              int32_t* budgets, int32_t* perm, float* curves, double* vsum,
                              void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(v, P));
  if (!scores || !budgets) return CERTKV_EINVAL;
  if (P.dtype == CERTKV_F32 && P.g.D != 64) return CERTKV_EUNSUPPORTED;
  TRY(check_budget(P, n_keep_host, alpha, steps));
  Bufs w;
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_ALLOCATE), ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  hipStream_t s = (hipStream_t)stream;
  int32_t* pm = perm ? perm : w.perm;
  float* cv = curves ? curves : w.curves;
  TRY(do_sort(P, scores, pm, w, s));
  TRY(do_curves(P, v, pm, cv, vsum, w, s));
  return do_allocate(P, cv, n_keep_host, alpha, steps, budgets, false, w, s);
}

certkv_status certkv_allocate_curves(const certkv_problem* p, const float* curves,
                                     const int32_t* n_keep_host, double alpha, int32_t steps,
                                     int32_t* budgets, void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  if (!curves || !budgets) return CERTKV_EINVAL;
  TRY(check_budget(P, n_keep_host, alpha, steps));
  Bufs w;
  TRY(check_ws(P, NEED_MINMAX, ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  return do_allocate(P, curves, n_keep_host, alpha, steps, budgets, true, w, (hipStream_t)stream);
}

certkv_status certkv_select(const certkv_problem* p, const float* scores, int32_t* budgets_io,
                            int32_t mode, double retain_mass, int64_t* kept_offsets,
                            int32_t* kept_idx, int64_t kept_capacity, uint8_t* kept_mask, void* ws,
                            size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  if (!scores || !budgets_io || !kept_offsets || !kept_idx || kept_capacity < 0)
    return CERTKV_EINVAL;
  if (mode != CERTKV_SELECT_BUDGET && mode != CERTKV_SELECT_COVERAGE) return CERTKV_EINVAL;
  if ((uintptr_t)kept_mask & 15u) return CERTKV_EINVAL;
  if (mode == CERTKV_SELECT_COVERAGE) {
    if (!(retain_mass > 0.0 && retain_mass <= 1.0)) return CERTKV_EINVAL;
    if (kept_capacity < (int64_t)P.g.L * P.g.H * P.g.T) return CERTKV_EINVAL;
  }
  Bufs w;
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_SELECT), ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  hipStream_t s = (hipStream_t)stream;
  TRY(do_sort(P, scores, w.perm, w, s));
  TRY(do_select(P, scores, w.keysA, w.perm, budgets_io, mode, retain_mass, kept_offsets, nullptr,
                kept_idx, kept_capacity, nullptr, s));
  if (kept_mask) TRY(run_mask(P.g, make_tabs(P, nullptr, 0.f), kept_offsets, kept_idx, kept_mask, s));
  return CERTKV_OK;
}

certkv_status certkv_tail_summary(const certkv_problem* p, const float* scores, certkv_tensor k,
                                  certkv_tensor v, const int64_t* kept_offsets,
                                  const int32_t* kept_idx, const double* ksum, const double* vsum,
                                  float* k_star, float* v_star, double* tail_mass, void* ws,
                                  size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(k, P));
  TRY(check_tensor(v, P));
  if (!scores || !kept_offsets || !kept_idx || !k_star || !v_star || !tail_mass)
    return CERTKV_EINVAL;
  Bufs w;
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_TAIL), ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  const bool comp = ksum && vsum;
  return do_tail(P, scores, k, v, kept_offsets, kept_idx, comp ? ksum : nullptr,
                 comp ? vsum : nullptr, k_star, v_star, tail_mass, nullptr, nullptr, nullptr, true,
                 false, false, w, (hipStream_t)stream);
}

certkv_status certkv_compact(const certkv_problem* p, certkv_tensor k, certkv_tensor v,
                             const int64_t* kept_offsets, const int32_t* kept_idx,
                             const float* k_star, const float* v_star, void* k_packed,
                             void* v_packed, int32_t* pos_packed, int64_t* packed_offsets,
                             void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(k, P));
  TRY(check_tensor(v, P));
  if (!kept_offsets || !kept_idx || !k_star || !v_star || !k_packed || !v_packed || !pos_packed ||
      !packed_offsets)
    return CERTKV_EINVAL;
  if (((uintptr_t)k_packed & 15u) || ((uintptr_t)v_packed & 15u)) return CERTKV_EINVAL;
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  hipStream_t s = (hipStream_t)stream;
  // packed_offsets[u] = kept_offsets[u] + u: recompute from the kept counts.
  Bufs w;
  TRY(run_packed_from_kept(P.U, P.g.slot, kept_offsets, packed_offsets, s));
  TRY(do_tail(P, nullptr, k, v, kept_offsets, kept_idx, nullptr, nullptr, const_cast<float*>(k_star),
              const_cast<float*>(v_star), nullptr, k_packed, v_packed, pos_packed, false, true,
              false, w, s));
  return CERTKV_OK;
}

// Decode partials: [rows][d] fp32 outputs, then (on a 256-byte boundary) the
// rows' (max, sum) pairs.
// A segment holds b_h <= n_b - 1 kept rows plus the slot row.
static int decode_rows_bound(const Plan& P, int32_t max_rows) {
  return (max_rows > 0 && max_rows < P.max_len) ? max_rows : P.max_len;
}

// Decode workspace: split partials (output rows, then (max, sum) pairs), the
// work-item list and its length, each 256-byte aligned.
struct DecodeWs {
  int nsplit;
  size_t ml_off, items_off, count_off, total;
};
static DecodeWs decode_ws_layout(const Plan& P, int32_t tq, int32_t max_rows) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  DecodeWs w;
  w.nsplit = decode_nsplit(decode_rows_bound(P, max_rows));
  const size_t rows = decode_partial_rows(P.U, w.nsplit, tq, P.g.G);
  w.ml_off = up(rows * (size_t)P.g.D * sizeof(float));
  w.items_off = up(w.ml_off + rows * sizeof(float2));
  w.count_off = up(w.items_off + (size_t)P.U * w.nsplit * sizeof(int2));
  w.total = w.count_off + 256;
  return w;
}

size_t certkv_decode_workspace_size(const certkv_problem* p, int32_t tq, int32_t max_rows) {
  Plan P;
  if (make_plan(p, &P) != CERTKV_OK || tq < 1 || max_rows < 0) return 0;
  return decode_ws_layout(P, tq, max_rows).total;
}

static certkv_status decode_impl(const certkv_problem* p, certkv_tensor q_new, int32_t tq,
                                 int32_t max_rows, const void* k_packed, const void* v_packed,
                                 const int64_t* packed_offsets, const DecodeClusters& cl,
                                 float* out, float* lse, void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  if (tq < 1 || max_rows < 0) return CERTKV_EINVAL;
  // Cluster terms stand for the evicted ranks; a packed segment that already
  // ends in the slot row (which carries the whole evicted tail) would count
  // that mass twice, so the clustered decode needs a no-slot problem.
  if (cl.m > 0 && P.g.slot) return CERTKV_EINVAL;
  if (P.dtype != CERTKV_BF16) return CERTKV_EUNSUPPORTED;
  if ((int64_t)tq * P.g.G > 512) return CERTKV_EUNSUPPORTED;
  if (!q_new.ptr || ((uintptr_t)q_new.ptr & 15u)) return CERTKV_EINVAL;
  if ((q_new.s_layer % 8) || (q_new.s_token % 8) || (q_new.s_head % 8)) return CERTKV_EINVAL;
  if (q_new.s_layer < 0 || q_new.s_token < 0 || q_new.s_head < 0) return CERTKV_EINVAL;
  if (!k_packed || !v_packed || !packed_offsets || !out) return CERTKV_EINVAL;
  if (((uintptr_t)k_packed & 15u) || ((uintptr_t)v_packed & 15u)) return CERTKV_EINVAL;
  const size_t need = certkv_decode_workspace_size(p, tq, max_rows);
  if (!ws) return CERTKV_EWORKSPACE;
  if (((uintptr_t)ws & 255u) != 0) return CERTKV_EINVAL;
  if (ws_bytes < need) return CERTKV_EWORKSPACE;
  const DecodeWs W = decode_ws_layout(P, tq, max_rows);
  if ((int64_t)P.U * W.nsplit > INT32_MAX) return CERTKV_EUNSUPPORTED;
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  DecodeArgs a;
  a.g = P.g;
  a.U = P.U;
  a.tq = tq;
  a.nsplit = W.nsplit;
  a.q = q_new;
  a.k_packed = k_packed;
  a.v_packed = v_packed;
  a.packed_offsets = packed_offsets;
  a.part_o = static_cast<float*>(ws);
  a.part_ml = reinterpret_cast<float2*>(static_cast<char*>(ws) + W.ml_off);
  a.items = reinterpret_cast<int2*>(static_cast<char*>(ws) + W.items_off);
  a.item_count = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + W.count_off);
  a.cl = cl;
  a.out = out;
  a.lse = lse;
  return run_decode(a, (hipStream_t)stream);
}

certkv_status certkv_decode(const certkv_problem* p, certkv_tensor q_new, int32_t tq,
                            int32_t max_rows, const void* k_packed, const void* v_packed,
                            const int64_t* packed_offsets, float* out, float* lse, void* ws,
                            size_t ws_bytes, void* stream) {
  DecodeClusters cl;
  memset(&cl, 0, sizeof(cl));
  return decode_impl(p, q_new, tq, max_rows, k_packed, v_packed, packed_offsets, cl, out, lse, ws,
                     ws_bytes, stream);
}

certkv_status certkv_decode_clustered(const certkv_problem* p, certkv_tensor q_new, int32_t tq,
                                      int32_t max_rows, const void* k_packed,
                                      const void* v_packed, const int64_t* packed_offsets,
                                      int32_t m, const void* cluster_k, const void* cluster_v,
                                      const int32_t* cluster_count, const float* cluster_rk,
                                      const float* cluster_rv, const float* kept_vmax,
                                      float* out, float* lse, float* bound, void* ws,
                                      size_t ws_bytes, void* stream) {
  if (m < 1 || m > 64) return CERTKV_EINVAL;
  if (!cluster_k || !cluster_v || !cluster_count || !cluster_rk || !cluster_rv || !kept_vmax)
    return CERTKV_EINVAL;
  DecodeClusters cl;
  cl.m = m;
  cl.kbar = static_cast<const uint16_t*>(cluster_k);
  cl.vbar = static_cast<const uint16_t*>(cluster_v);
  cl.count = cluster_count;
  cl.rk = cluster_rk;
  cl.rv = cluster_rv;
  cl.vmax_kept = kept_vmax;
  cl.bound = bound;
  return decode_impl(p, q_new, tq, max_rows, k_packed, v_packed, packed_offsets, cl, out, lse, ws,
                     ws_bytes, stream);
}

certkv_status certkv_cluster_tail(const certkv_problem* p, certkv_tensor k, certkv_tensor v,
                                  const int32_t* perm, const int32_t* budgets, int32_t m,
                                  void* cluster_k, void* cluster_v, int32_t* cluster_count,
                                  float* cluster_rk, float* cluster_rv, float* kept_vmax,
                                  void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(k, P));
  TRY(check_tensor(v, P));
  if (m < 1 || m > 64) return CERTKV_EINVAL;
  // the summaries replace the single slot: the problem must have none
  if (P.g.slot) return CERTKV_EINVAL;
  if (!perm || !budgets || !cluster_k || !cluster_v || !cluster_count || !cluster_rk ||
      !cluster_rv || !kept_vmax)
    return CERTKV_EINVAL;
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  ClusterArgs a;
  a.g = P.g;
  a.dtype = P.dtype;
  a.m = m;
  a.perm = perm;
  a.budgets = budgets;
  a.k = k;
  a.v = v;
  a.kbar = cluster_k;
  a.vbar = cluster_v;
  a.count = cluster_count;
  a.rk = cluster_rk;
  a.rv = cluster_rv;
  a.vmax_kept = kept_vmax;
  TRY(run_clusters_clear(kept_vmax, P.U, (hipStream_t)stream));
  for (const SeqTab& t : make_tabs(P, nullptr, 0.0)) TRY(run_clusters(a, t, (hipStream_t)stream));
  return CERTKV_OK;
}

certkv_status certkv_compress(const certkv_problem* p, certkv_tensor q_win, certkv_tensor k,
                              certkv_tensor v, const float* lse_in, const int32_t* n_keep_host,
                              double alpha, int32_t steps, const certkv_outputs* out, void* ws,
                              size_t ws_bytes, void* stream) {
  Plan P;
  TRY(make_plan(p, &P));
  TRY(check_tensor(q_win, P));
  TRY(check_tensor(k, P));
  TRY(check_tensor(v, P));
  if (!out || !out->scores || !out->budgets || !out->kept_offsets || !out->kept_idx ||
      !out->k_star || !out->v_star || !out->tail_mass || !out->k_packed || !out->v_packed ||
      !out->pos_packed || !out->packed_offsets)
    return CERTKV_EINVAL;
  if (((uintptr_t)out->k_packed & 15u) || ((uintptr_t)out->v_packed & 15u)) return CERTKV_EINVAL;
  if ((uintptr_t)out->kept_mask & 15u) return CERTKV_EINVAL;
  if (P.dtype == CERTKV_F32 && P.g.D != 64) return CERTKV_EUNSUPPORTED;
  TRY(check_budget(P, n_keep_host, alpha, steps));
  Bufs w;
  TRY(check_ws(P, stage_needs(CERTKV_STAGE_COMPRESS), ws, ws_bytes, &w));
  if (p->flags & CERTKV_DRY_RUN) return CERTKV_OK;
  hipStream_t s = (hipStream_t)stream;
  int32_t* pm = out->perm ? out->perm : w.perm;
  float* cv = out->curves ? out->curves : w.curves;
  int64_t cap = 0;
  for (int b = 0; b < P.g.B; ++b)
    cap += (int64_t)P.g.H * n_keep_host[b] - (P.g.slot ? P.g.H : 0);
  cap *= P.g.L;
  TRY(do_score(P, q_win, k, lse_in, out->scores, w.ksum, out->lse, w, s));
  TRY(do_sort(P, out->scores, pm, w, s));
  TRY(do_curves(P, v, pm, cv, w.vsum, w, s));
  TRY(do_allocate(P, cv, n_keep_host, alpha, steps, out->budgets, false, w, s, out->alloc_stats));
  TRY(do_select(P, out->scores, w.keysA, pm, out->budgets, CERTKV_SELECT_BUDGET, 0.0,
                out->kept_offsets, out->packed_offsets, out->kept_idx, cap, &w, s));
  TRY(do_tail(P, out->scores, k, v, out->kept_offsets, out->kept_idx, w.ksum, w.vsum, out->k_star,
              out->v_star, out->tail_mass, out->k_packed, out->v_packed, out->pos_packed, true, true,
              true, w, s));
  if (out->kept_mask)
    TRY(run_mask(P.g, make_tabs(P, nullptr, 0.f), out->kept_offsets, out->kept_idx, out->kept_mask,
                 s));
  return CERTKV_OK;
}

certkv_status certkv_profile_enable(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = enable != 0;
  return CERTKV_OK;
}

void certkv_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    if (r.a) hipEventSynchronize(r.a);
    if (r.b) hipEventSynchronize(r.b);
    if (r.a) g_pool.push_back(r.a);
    if (r.b) g_pool.push_back(r.b);
  }
  g_prof.clear();
}

int32_t certkv_profile_read(char (*names)[64], int64_t* counts, double* total_ms,
                            int32_t max_entries) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  std::vector<std::string> nm;
  std::vector<int64_t> cnt;
  std::vector<double> ms;
  for (auto& r : g_prof) {
    if (!r.a || !r.b) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) continue;
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) continue;
    size_t i = 0;
    for (; i < nm.size(); ++i)
      if (nm[i] == r.name) break;
    if (i == nm.size()) {
      nm.push_back(r.name);
      cnt.push_back(0);
      ms.push_back(0.0);
    }
    cnt[i] += 1;
    ms[i] += t;
  }
  const int32_t k = (int32_t)nm.size();
  for (int32_t i = 0; i < k && i < max_entries; ++i) {
    if (names) {
      strncpy(names[i], nm[i].c_str(), 63);
      names[i][63] = 0;
    }
    if (counts) counts[i] = cnt[i];
    if (total_ms) total_ms[i] = ms[i];
  }
  return k;
}

}  // extern "C"
