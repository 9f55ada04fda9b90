// libdif C ABI: host-side runtime around the gfx950 kernels.
//
// Owns no device memory.  A plan is host metadata (index tables, kept
// widths, pointers) over caller-provided device memory that holds the
// step's compacted weights; the workspace is carved into the activation
// buffers of one block / one step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dif.h"
#include "kernels.h"

using dif::bf16;

namespace {

thread_local std::string g_err;

dif_status fail(dif_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(DIF_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define DIF_TRY(expr)                 \
  do {                                \
    dif_status s_ = (expr);           \
    if (s_ != DIF_OK) return s_;      \
  } while (0)

#define GUARD_BEGIN try {
#define GUARD_END                                                  \
  }                                                                \
  catch (const std::exception& ex) {                               \
    return fail(DIF_E_ARG, "internal error: %s", ex.what());       \
  }                                                                \
  catch (...) {                                                    \
    return fail(DIF_E_ARG, "internal error");                      \
  }

inline size_t align256(size_t n) { return (n + 255) & ~size_t(255); }
inline int64_t round_up(int64_t n, int64_t m) { return (n + m - 1) / m * m; }
inline size_t esize(int dtype) { return dtype == DIF_BF16 ? 2 : 4; }

// ---------------------------------------------------------------------------
// kernel timing
// ---------------------------------------------------------------------------
enum ProfKind {
  PK_GEMM_QKV = 0, PK_ATTN_SELF, PK_GEMM_SELF_OUT, PK_GEMM_CROSS_Q, PK_GEMM_CROSS_KV,
  PK_ATTN_CROSS, PK_GEMM_CROSS_OUT, PK_GEMM_FFN1, PK_GEMM_FFN2, PK_NORM, PK_QK_NORM,
  PK_TRANSPOSE, PK_TIME_EMBED, PK_GEMM_IO, PK_GATHER, PK_ELEMENTWISE
};
const char* kKindNames[DIF_PROF_KINDS] = {
    "gemm_qkv", "attn_self", "gemm_self_out", "gemm_cross_q", "gemm_cross_kv", "attn_cross",
    "gemm_cross_out", "gemm_ffn1", "gemm_ffn2", "norm", "qk_norm_rope", "transpose_v",
    "time_embed", "gemm_io", "gather", "elementwise"};

struct ProfRec {
  int kind;
  hipEvent_t a, b;
  double flops, bytes;
};
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  hipEvent_t take() {
    if (used < pool.size()) return pool[used++];
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    pool.push_back(e);
    ++used;
    return e;
  }
};
Profiler g_prof;

// Brackets the launches issued in its scope with events on `stream`.
class ProfScope {
 public:
  ProfScope(int kind, hipStream_t s, double flops, double bytes)
      : kind_(kind), s_(s), flops_(flops), bytes_(bytes) {
    if (!g_prof.on) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    a_ = g_prof.take();
    // a launch whose start event cannot be recorded is left out of the timing
    if (a_ && hipEventRecord(a_, s_) != hipSuccess) a_ = nullptr;
  }
  ~ProfScope() {
    if (!a_) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    hipEvent_t b = g_prof.take();
    if (!b || hipEventRecord(b, s_) != hipSuccess) return;
    g_prof.recs.push_back({kind_, a_, b, flops_, bytes_});
  }

 private:
  int kind_;
  hipStream_t s_;
  double flops_, bytes_;
  hipEvent_t a_ = nullptr;
};

// ---------------------------------------------------------------------------
// validation (host only)
// ---------------------------------------------------------------------------
dif_status check_config(const dif_config* c) {
  if (!c) return fail(DIF_E_ARG, "config is null");
  if (c->dim <= 0 || c->n_heads <= 0 || c->head_dim <= 0 || c->ffn_dim <= 0 || c->n_layers <= 0 ||
      c->patch_dim <= 0 || c->freq_dim <= 0 || c->max_text_len <= 0)
    return fail(DIF_E_SHAPE, "non-positive size in config");
  if (c->grid_f <= 0 || c->grid_h <= 0 || c->grid_w <= 0)
    return fail(DIF_E_SHAPE, "non-positive token grid");
  if ((int64_t)c->grid_f * c->grid_h * c->grid_w > (1 << 24))
    return fail(DIF_E_SHAPE, "token grid too large");
  if (c->dtype != DIF_BF16 && c->dtype != DIF_F32) return fail(DIF_E_ARG, "unknown dtype %d", c->dtype);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DIF_E_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", c->head_dim);
  if ((int64_t)c->n_heads * c->head_dim != c->dim)
    return fail(DIF_E_SHAPE, "dim %d != n_heads %d * head_dim %d", c->dim, c->n_heads, c->head_dim);
  const int max_dim = c->dtype == DIF_BF16 ? 8192 : 4096;
  if (c->dim % 64 != 0 || c->dim > max_dim)
    return fail(DIF_E_SHAPE, "dim %d must be a multiple of 64 and <= %d", c->dim, max_dim);
  if (c->patch_dim % 64 != 0) return fail(DIF_E_SHAPE, "patch_dim %d must be a multiple of 64", c->patch_dim);
  if (c->freq_dim % 16 != 0) return fail(DIF_E_SHAPE, "freq_dim %d must be a multiple of 16", c->freq_dim);
  if (c->ffn_dim > (1 << 20)) return fail(DIF_E_SHAPE, "ffn_dim too large");
  if (!(c->eps > 0.f) || !(c->rope_theta > 0.f)) return fail(DIF_E_ARG, "eps and rope_theta must be > 0");
  return DIF_OK;
}

// Indexed plans read 16-byte chunks of W2's rows in place: the FFN width
// must be whole chunks for either dtype, and one layer's chunk table must
// fit the GEMM's LDS table (8192 chunks).
dif_status check_plan_kind(const dif_config* c, int32_t kind) {
  if (kind == DIF_PLAN_COMPACT) return DIF_OK;
  if (kind != DIF_PLAN_INDEXED) return fail(DIF_E_ARG, "unknown plan kind %d", kind);
  if (c->ffn_dim % 8 != 0)
    return fail(DIF_E_UNSUPPORTED, "indexed plan: ffn_dim %d must be a multiple of 8", c->ffn_dim);
  const int vec = (int)(16 / esize(c->dtype));
  if ((int64_t)round_up(c->ffn_dim, 64) / vec > 8192)
    return fail(DIF_E_UNSUPPORTED, "indexed plan: ffn_dim %d too large", c->ffn_dim);
  return DIF_OK;
}

dif_status check_masks(const dif_config* c, const dif_step_masks* m) {
  if (!m || !m->block_keep || !m->self_head_keep || !m->cross_head_keep || !m->ffn_keep)
    return fail(DIF_E_MASK, "mask pointer is null");
  auto bad = [](const uint8_t* p, int64_t n) {
    for (int64_t i = 0; i < n; ++i)
      if (p[i] > 1) return i;
    return (int64_t)-1;
  };
  int64_t i;
  if ((i = bad(m->block_keep, c->n_layers)) >= 0) return fail(DIF_E_MASK, "block_keep[%lld] not 0/1", (long long)i);
  if ((i = bad(m->self_head_keep, (int64_t)c->n_layers * c->n_heads)) >= 0)
    return fail(DIF_E_MASK, "self_head_keep[%lld] not 0/1", (long long)i);
  if ((i = bad(m->cross_head_keep, (int64_t)c->n_layers * c->n_heads)) >= 0)
    return fail(DIF_E_MASK, "cross_head_keep[%lld] not 0/1", (long long)i);
  if ((i = bad(m->ffn_keep, (int64_t)c->n_layers * c->ffn_dim)) >= 0)
    return fail(DIF_E_MASK, "ffn_keep[%lld] not 0/1", (long long)i);
  return DIF_OK;
}

// ---------------------------------------------------------------------------
// plan layout
// ---------------------------------------------------------------------------
struct LayerPlan {
  dif_layer_info info{};
  // offsets into plan memory, resolved to pointers once plan_mem is known
  size_t o_wqkv = 0, o_bqkv = 0, o_gq = 0, o_gk = 0, o_wo = 0;
  size_t o_wcq = 0, o_bcq = 0, o_gcq = 0, o_gck = 0, o_wckv = 0, o_bckv = 0, o_wco = 0;
  size_t o_w1 = 0, o_b1 = 0, o_w2 = 0;
  size_t o_idx_self = 0, o_idx_cross = 0, o_idx_ffn = 0;   // device index tables
  size_t h_idx_self = 0, h_idx_cross = 0, h_idx_ffn = 0;   // offsets into host_idx
  // indexed plans: K-chunk tables (16-byte chunks of the union's reduction axis)
  size_t o_kch_self = 0, o_kch_cross = 0, o_kch_ffn = 0;
  size_t h_kch_self = 0, h_kch_cross = 0, h_kch_ffn = 0;
  char* base = nullptr;
  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(base + off); }
};

struct Layout {
  bool indexed = false;
  std::vector<LayerPlan> layers;
  std::vector<int32_t> host_idx;
  size_t o_rope = 0, n_rope = 0, o_idx = 0, total = 0;
};

struct Carve {
  size_t off = 0;
  size_t take(size_t n) {
    const size_t o = off;
    off = align256(off + n);
    return o;
  }
};

void rope_pairs(int dh, int* jt, int* jh, int* jw) {
  const int dhw = 2 * (dh / 6);
  *jt = (dh - 2 * dhw) / 2;
  *jh = dhw / 2;
  *jw = dhw / 2;
}

}  // namespace

struct dif_model {
  dif_config cfg;
  dif_weights w;
  std::vector<dif_layer_weights> layers;
  int ncu = 0;   // compute units of the device the model was created on
};

struct dif_plan {
  const dif_model* model = nullptr;
  int32_t step = 0;
  float t_s = 0.f;       // the timestep this structure belongs to
  int32_t flags = 0;     // DIF_PLAN_ANY_T: any timestep accepted
  Layout lay;
  std::vector<float> host_rope;
  char* mem = nullptr;
  size_t bytes = 0;
  dif::RopeDesc rope{};
};

namespace {

// Index tables of one step structure (Sec. 4.3, I_t).
//   compact plan: kept rows (heads: h*dh entries; FFN: kept channels, -1 up
//     to the 64-padded width), then the compacted weights carved after them.
//   indexed plan: the same head row tables plus, per table, the 16-byte
//     chunks of the union's reduction axis (dh/VEC per head); the FFN keeps
//     whole VEC-channel chunks that hold at least one kept channel, with -1
//     for the dropped channels inside them and for the padding to 64.
//     No weights are copied.
Layout build_layout(const dif_model* m, const dif_step_masks* mk, bool indexed) {
  const dif_config& c = m->cfg;
  const size_t es = esize(c.dtype);
  const int vec = (int)(16 / es);
  const int D = c.dim, dh = c.head_dim, H = c.n_heads, F = c.ffn_dim;
  Layout L;
  L.indexed = indexed;
  Carve cv;
  int jt, jh, jw;
  rope_pairs(dh, &jt, &jh, &jw);
  L.n_rope = (size_t)c.grid_f * jt + (size_t)c.grid_h * jh + (size_t)c.grid_w * jw;
  L.o_rope = cv.take(L.n_rope * 2 * sizeof(float));
  L.layers.resize(c.n_layers);
  std::vector<int32_t>& ix = L.host_idx;
  auto head_rows = [&](const uint8_t* keep) {
    for (int i = 0; i < H; ++i)
      if (keep[i])
        for (int d = 0; d < dh; ++d) ix.push_back(i * dh + d);
  };
  auto head_chunks = [&](const uint8_t* keep) {
    for (int i = 0; i < H; ++i)
      if (keep[i])
        for (int q = 0; q < dh / vec; ++q) ix.push_back((i * dh) / vec + q);
  };
  for (int l = 0; l < c.n_layers; ++l) {
    LayerPlan& lp = L.layers[l];
    lp.info.block_keep = mk->block_keep[l];
    const uint8_t* ks = mk->self_head_keep + (size_t)l * H;
    const uint8_t* kc = mk->cross_head_keep + (size_t)l * H;
    const uint8_t* kf = mk->ffn_keep + (size_t)l * F;
    int h = 0, hc = 0, f = 0, touched = 0;
    for (int i = 0; i < H; ++i) {
      h += ks[i];
      hc += kc[i];
    }
    for (int i = 0; i < F; ++i) f += kf[i];
    for (int t = 0; indexed && t < F / vec; ++t) {
      bool any = false;
      for (int e = 0; e < vec; ++e) any = any || kf[t * vec + e];
      touched += any;
    }
    lp.info.self_heads = h;
    lp.info.cross_heads = hc;
    lp.info.ffn_channels = f;
    lp.info.ffn_padded = (int)round_up(indexed ? (int64_t)touched * vec : f, 64);
    if (!lp.info.block_keep) continue;
    const int fp = lp.info.ffn_padded;
    lp.h_idx_self = ix.size();
    head_rows(ks);
    lp.h_idx_cross = ix.size();
    head_rows(kc);
    lp.h_idx_ffn = ix.size();
    if (!indexed) {
      for (int i = 0; i < F; ++i)
        if (kf[i]) ix.push_back(i);
    } else {
      for (int t = 0; t < F / vec; ++t) {
        bool any = false;
        for (int e = 0; e < vec; ++e) any = any || kf[t * vec + e];
        if (any)
          for (int e = 0; e < vec; ++e) ix.push_back(kf[t * vec + e] ? t * vec + e : -1);
      }
    }
    while ((int64_t)(ix.size() - lp.h_idx_ffn) < fp) ix.push_back(-1);
    if (indexed) {
      lp.h_kch_self = ix.size();
      head_chunks(ks);
      lp.h_kch_cross = ix.size();
      head_chunks(kc);
      lp.h_kch_ffn = ix.size();
      for (int t = 0; t < F / vec; ++t) {
        bool any = false;
        for (int e = 0; e < vec; ++e) any = any || kf[t * vec + e];
        if (any) ix.push_back(t);
      }
      while ((int64_t)(ix.size() - lp.h_kch_ffn) < fp / vec) ix.push_back(-1);
    }
  }
  L.o_idx = cv.take(ix.size() * sizeof(int32_t));
  for (int l = 0; l < c.n_layers; ++l) {
    LayerPlan& lp = L.layers[l];
    if (!lp.info.block_keep) continue;
    const size_t a = (size_t)lp.info.self_heads * dh, ac = (size_t)lp.info.cross_heads * dh;
    const size_t fp = lp.info.ffn_padded;
    lp.o_idx_self = L.o_idx + lp.h_idx_self * sizeof(int32_t);
    lp.o_idx_cross = L.o_idx + lp.h_idx_cross * sizeof(int32_t);
    lp.o_idx_ffn = L.o_idx + lp.h_idx_ffn * sizeof(int32_t);
    if (indexed) {
      lp.o_kch_self = L.o_idx + lp.h_kch_self * sizeof(int32_t);
      lp.o_kch_cross = L.o_idx + lp.h_kch_cross * sizeof(int32_t);
      lp.o_kch_ffn = L.o_idx + lp.h_kch_ffn * sizeof(int32_t);
      continue;
    }
    lp.o_wqkv = cv.take(3 * a * D * es);
    lp.o_bqkv = cv.take(3 * a * 4);
    lp.o_gq = cv.take(a * 4);
    lp.o_gk = cv.take(a * 4);
    lp.o_wo = cv.take((size_t)D * a * es);
    lp.o_wcq = cv.take(ac * D * es);
    lp.o_bcq = cv.take(ac * 4);
    lp.o_gcq = cv.take(ac * 4);
    lp.o_gck = cv.take(ac * 4);
    lp.o_wckv = cv.take(2 * ac * D * es);
    lp.o_bckv = cv.take(2 * ac * 4);
    lp.o_wco = cv.take((size_t)D * ac * es);
    lp.o_w1 = cv.take(fp * D * es);
    lp.o_b1 = cv.take(fp * 4);
    lp.o_w2 = cv.take((size_t)D * fp * es);
  }
  L.total = cv.off;
  return L;
}

// ---------------------------------------------------------------------------
// workspace layout
// ---------------------------------------------------------------------------
struct WsLayout {
  size_t xn, big, vt, o, ckv, cvt, x, zc, e, e0, t1, t2, emb, part, part_bytes, total;
  int64_t ldvt, ldcvt;
};

WsLayout ws_layout(const dif_config& c, int B, int L, int Lc) {
  const size_t es = esize(c.dtype);
  const size_t M = (size_t)B * L, Mc = (size_t)B * Lc, D = c.dim;
  const size_t Fp = round_up(c.ffn_dim, 64);
  WsLayout w{};
  w.ldvt = round_up(L, 64);
  w.ldcvt = round_up(Lc, 64);
  Carve cv;
  w.xn = cv.take(M * D * es);
  w.big = cv.take(M * std::max(3 * D, Fp) * es);
  w.vt = cv.take((size_t)B * D * w.ldvt * es);
  w.o = cv.take(M * D * es);
  w.ckv = cv.take(Mc * 2 * D * es);
  w.cvt = cv.take((size_t)B * D * w.ldcvt * es);
  w.x = cv.take(M * D * es);
  w.zc = cv.take(M * c.patch_dim * es);
  w.e = cv.take(D * 4);
  w.e0 = cv.take(6 * D * 4);
  w.t1 = cv.take(std::max<size_t>(D, c.freq_dim) * 4);
  w.t2 = cv.take(std::max<size_t>(D, c.freq_dim) * 4);
  w.emb = cv.take(c.freq_dim * 4);
  // self-attention key splits: bf16 self-attention over long keys only
  const bool split = c.dtype == DIF_BF16 && L >= dif::kAttnLongKeys;
  w.part = cv.take(split ? dif::attention_split_bytes(c.head_dim) : 0);
  w.part_bytes = split ? dif::attention_split_bytes(c.head_dim) : 0;
  w.total = cv.off;
  return w;
}

// Cross-attention text cache: per layer, the text tokens' keys before their
// RMSNorm, k = ctx W_ck^T + b_ck [B*Lc, D], and values transposed,
// v^T [B, D, ldcvt] (zero past Lc), for all heads; then one [B*Lc, D]
// staging buffer used while building.
struct TextLayout {
  size_t k_bytes, vt_bytes, per_layer, stage, total;
  int64_t ldcvt;
  size_t k(int l) const { return (size_t)l * per_layer; }
  size_t vt(int l) const { return (size_t)l * per_layer + k_bytes; }
};

TextLayout text_layout(const dif_config& c, int B, int Lc) {
  const size_t es = esize(c.dtype), Mc = (size_t)B * Lc, D = c.dim;
  TextLayout t{};
  t.ldcvt = round_up(Lc, 64);
  t.k_bytes = align256(Mc * D * es);
  t.vt_bytes = align256((size_t)B * D * t.ldcvt * es);
  t.per_layer = t.k_bytes + t.vt_bytes;
  t.stage = (size_t)c.n_layers * t.per_layer;
  t.total = t.stage + align256(Mc * D * es);
  return t;
}

dif_status check_text(const dif_config& c, int B, int Lc) {
  if (B <= 0) return fail(DIF_E_SHAPE, "B must be >= 1");
  if (Lc < 1 || Lc > c.max_text_len) return fail(DIF_E_SHAPE, "Lc = %d outside [1, %d]", Lc, c.max_text_len);
  if ((int64_t)B * Lc * c.dim > ((int64_t)1 << 31) / 2) return fail(DIF_E_SHAPE, "B * Lc too large");
  return DIF_OK;
}

dif_status check_cache(const TextLayout& t, const void* cache, size_t bytes) {
  if (!cache) return fail(DIF_E_ARG, "text cache is null");
  if (reinterpret_cast<uintptr_t>(cache) % 256) return fail(DIF_E_ARG, "text cache not 256-byte aligned");
  if (bytes < t.total) return fail(DIF_E_WORKSPACE, "text cache %zu bytes < required %zu", bytes, t.total);
  return DIF_OK;
}

dif_status check_ws(const WsLayout& w, const void* ws, size_t bytes) {
  if (!ws) return fail(DIF_E_WORKSPACE, "workspace is null");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(DIF_E_WORKSPACE, "workspace not 256-byte aligned");
  if (bytes < w.total)
    return fail(DIF_E_WORKSPACE, "workspace %zu bytes < required %zu", bytes, w.total);
  return DIF_OK;
}

// ---------------------------------------------------------------------------
// launches with timing
// ---------------------------------------------------------------------------
template <typename T, typename OutT>
dif_status gemm(int kind, const T* A, int64_t lda, const T* Bm, int64_t ldb, OutT* C, int64_t ldc,
                int M, int N, int K, int epi, const float* bias, const float* g0, const float* g1,
                hipStream_t s, const dif::GemmGather* gather = nullptr,
                const dif::GemmVt* vt = nullptr) {
  if (M <= 0 || N <= 0) return DIF_OK;
  const double es = sizeof(T);
  const double Nt = (double)N * (gather ? gather->nseg : 1);   // all segments
  const double bytes = ((double)M * K + Nt * K) * es + (double)M * Nt * sizeof(OutT) *
                                                          (epi == dif::EPI_RESIDUAL ? 2 : 1);
  ProfScope ps(kind, s, 2.0 * M * Nt * (double)K, bytes);
  HIP_TRY((dif::launch_gemm<T, OutT>(A, lda, Bm, ldb, C, ldc, M, N, K, epi, bias, g0, g1, s, gather,
                                     vt)));
  return DIF_OK;
}

template <typename T>
dif_status attention(int kind, int dh, const T* Q, int64_t ldq, const T* K, int64_t ldk,
                     const T* Vt, int64_t ldvt, T* O, int64_t ldo, int B, int Lq, int Lk, int H,
                     hipStream_t s, bool q_scaled = false, float* split_part = nullptr,
                     int ncu = 0) {
  if (H <= 0) return DIF_OK;
  const double flops = 4.0 * B * (double)Lq * Lk * dh * H;
  const double bytes = (double)B * (2.0 * Lq + 2.0 * Lk) * H * dh * sizeof(T);
  ProfScope ps(kind, s, flops, bytes);
  HIP_TRY(dif::launch_attention<T>(dh, Q, ldq, K, ldk, Vt, ldvt, O, ldo, B, Lq, Lk, H, s, q_scaled,
                                   split_part, ncu));
  return DIF_OK;
}

// ---------------------------------------------------------------------------
// plan construction
// ---------------------------------------------------------------------------
template <typename T>
dif_status gather_layer(const dif_model* m, int l, const LayerPlan& lp, hipStream_t s) {
  const dif_config& c = m->cfg;
  const dif_layer_weights& W = m->layers[l];
  const int D = c.dim, dh = c.head_dim, F = c.ffn_dim;
  const int a = lp.info.self_heads * dh, ac = lp.info.cross_heads * dh, fp = lp.info.ffn_padded;
  const int32_t* is = lp.at<int32_t>(lp.o_idx_self);
  const int32_t* ic = lp.at<int32_t>(lp.o_idx_cross);
  const int32_t* iff = lp.at<int32_t>(lp.o_idx_ffn);
  const size_t es = sizeof(T);
  ProfScope ps(PK_GATHER, s, 0.0,
               2.0 * es * ((3.0 * a + 2.0 * ac) * D + (double)a * D + (double)ac * D + 2.0 * fp * D + ac * (double)D));
  T* wqkv = lp.at<T>(lp.o_wqkv);
  HIP_TRY(dif::launch_gather<T>((const T*)W.self_wq, D, wqkv, D, a, D, is, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.self_wk, D, wqkv + (size_t)a * D, D, a, D, is, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.self_wv, D, wqkv + (size_t)2 * a * D, D, a, D, is, nullptr, s));
  float* bqkv = lp.at<float>(lp.o_bqkv);
  HIP_TRY(dif::launch_gather<float>(W.self_bq, 1, bqkv, 1, a, 1, is, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.self_bk, 1, bqkv + a, 1, a, 1, is, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.self_bv, 1, bqkv + 2 * a, 1, a, 1, is, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.self_gq, 1, lp.at<float>(lp.o_gq), 1, a, 1, is, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.self_gk, 1, lp.at<float>(lp.o_gk), 1, a, 1, is, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.self_wo, D, lp.at<T>(lp.o_wo), a, D, a, nullptr, is, s));

  HIP_TRY(dif::launch_gather<T>((const T*)W.cross_wq, D, lp.at<T>(lp.o_wcq), D, ac, D, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.cross_bq, 1, lp.at<float>(lp.o_bcq), 1, ac, 1, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.cross_gq, 1, lp.at<float>(lp.o_gcq), 1, ac, 1, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.cross_gk, 1, lp.at<float>(lp.o_gck), 1, ac, 1, ic, nullptr, s));
  T* wckv = lp.at<T>(lp.o_wckv);
  HIP_TRY(dif::launch_gather<T>((const T*)W.cross_wk, D, wckv, D, ac, D, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.cross_wv, D, wckv + (size_t)ac * D, D, ac, D, ic, nullptr, s));
  float* bckv = lp.at<float>(lp.o_bckv);
  HIP_TRY(dif::launch_gather<float>(W.cross_bk, 1, bckv, 1, ac, 1, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.cross_bv, 1, bckv + ac, 1, ac, 1, ic, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.cross_wo, D, lp.at<T>(lp.o_wco), ac, D, ac, nullptr, ic, s));

  HIP_TRY(dif::launch_gather<T>((const T*)W.ffn_w1, D, lp.at<T>(lp.o_w1), D, fp, D, iff, nullptr, s));
  HIP_TRY(dif::launch_gather<float>(W.ffn_b1, 1, lp.at<float>(lp.o_b1), 1, fp, 1, iff, nullptr, s));
  HIP_TRY(dif::launch_gather<T>((const T*)W.ffn_w2, F, lp.at<T>(lp.o_w2), fp, D, fp, nullptr, iff, s));
  return DIF_OK;
}

// ---------------------------------------------------------------------------
// one block
// ---------------------------------------------------------------------------
template <typename T>
dif_status block_impl(const dif_plan* plan, int layer, T* x, const T* ctx, const float* e0, int B,
                      int L, int Lc, char* ws, const WsLayout& wl, hipStream_t s,
                      const T* tk = nullptr, const T* tvt = nullptr) {
  const dif_model* m = plan->model;
  const dif_config& c = m->cfg;
  const LayerPlan& lp = plan->lay.layers[layer];
  if (!lp.info.block_keep) return DIF_OK;
  const dif_layer_weights& W = m->layers[layer];
  const int D = c.dim, dh = c.head_dim;
  const int M = B * L, Mc = B * Lc;
  const int a = lp.info.self_heads * dh, ac = lp.info.cross_heads * dh, fp = lp.info.ffn_padded;
  const float* mod = W.mod;
  const float inv_d = 1.f / (float)D;
  // queries leave QK-norm already multiplied by the softmax scale in base 2
  const float q_scale = (float)(1.4426950408889634 / std::sqrt((double)dh));
  T* xn = reinterpret_cast<T*>(ws + wl.xn);
  T* big = reinterpret_cast<T*>(ws + wl.big);
  T* vt = reinterpret_cast<T*>(ws + wl.vt);
  T* o = reinterpret_cast<T*>(ws + wl.o);
  T* ckv = reinterpret_cast<T*>(ws + wl.ckv);
  T* cvt = reinterpret_cast<T*>(ws + wl.cvt);
  const double es = sizeof(T);

  // self-attention: LN + AdaLN(shift1, scale1)
  {
    ProfScope ps(PK_NORM, s, 0, 2.0 * M * D * es);
    HIP_TRY(dif::launch_norm<T>(x, xn, M, D, 0, mod, e0, mod + D, e0 + D, c.eps, s));
  }
  // Compact plans read the step's gathered weights; indexed plans read the
  // union weights through the tables (rows for output widths, 16-byte K
  // chunks for reduction widths).
  const bool ix = plan->lay.indexed;
  const int32_t* rs = lp.at<int32_t>(lp.o_idx_self);
  const int32_t* rc = lp.at<int32_t>(lp.o_idx_cross);
  const int32_t* rf = lp.at<int32_t>(lp.o_idx_ffn);
  const dif::GemmGather g_self_rows{rs, nullptr, D}, g_cross_rows{rc, nullptr, D},
      g_ffn_rows{rf, nullptr, c.ffn_dim};
  const dif::GemmGather g_self_k{nullptr, lp.at<int32_t>(lp.o_kch_self), 0},
      g_cross_k{nullptr, lp.at<int32_t>(lp.o_kch_cross), 0},
      g_ffn_k{nullptr, lp.at<int32_t>(lp.o_kch_ffn), 0};
  if (a > 0) {
    // q and k go to `big` (row-major, for QK-norm in place); v is written
    // transposed into vt [B, a, ldvt] by the same launch, as attention reads
    // it, when the v columns start on a GEMM tile (always for head width 128
    // and for indexed plans, where v is a launch segment of its own); else v
    // is stored with q and k and transposed by its own kernel
    const bool vt_in_gemm = ix || (2 * a) % 256 == 0;
    const dif::GemmVt vtd{vt, wl.ldvt, 2 * a, a, L};
    if (ix) {
      dif::GemmGather g = g_self_rows;
      g.nseg = 3;
      g.seg_b[0] = W.self_wk;
      g.seg_b[1] = W.self_wv;
      g.seg_bias[0] = W.self_bk;
      g.seg_bias[1] = W.self_bv;
      DIF_TRY((gemm<T, T>(PK_GEMM_QKV, xn, D, (const T*)W.self_wq, D, big, 3 * a, M, a, D,
                          dif::EPI_STORE, W.self_bq, nullptr, nullptr, s, &g, &vtd)));
    } else {
      DIF_TRY((gemm<T, T>(PK_GEMM_QKV, xn, D, lp.at<T>(lp.o_wqkv), D, big, 3 * a, M, 3 * a, D,
                          dif::EPI_STORE, lp.at<float>(lp.o_bqkv), nullptr, nullptr, s, nullptr,
                          vt_in_gemm ? &vtd : nullptr)));
    }
    {
      ProfScope ps(PK_QK_NORM, s, 0, 4.0 * M * a * es);
      dif::RopeDesc rd = plan->rope;
      rd.L = L;
      HIP_TRY(dif::launch_qk_norm<T>(big, 3 * a, M, a, 2, 0, a, ix ? W.self_gq : lp.at<float>(lp.o_gq),
                                     ix ? W.self_gk : lp.at<float>(lp.o_gk), inv_d, c.eps, &rd, s,
                                     ix ? rs : nullptr, q_scale));
    }
    if (!vt_in_gemm) {
      ProfScope ps(PK_TRANSPOSE, s, 0, 2.0 * M * a * es);
      HIP_TRY(dif::launch_transpose_vt<T>(big + 2 * a, 3 * a, a, B, L, vt, wl.ldvt, s));
    }
    DIF_TRY(attention<T>(PK_ATTN_SELF, dh, big, 3 * a, big + a, 3 * a, vt, wl.ldvt, o, a, B, L, L,
                         lp.info.self_heads, s, true,
                         wl.part_bytes ? reinterpret_cast<float*>(ws + wl.part) : nullptr, m->ncu));
  }
  if (ix)
    DIF_TRY((gemm<T, T>(PK_GEMM_SELF_OUT, o, std::max(a, 8), (const T*)W.self_wo, D, x, D, M, D, a,
                        dif::EPI_RESIDUAL, W.self_bo, mod + 2 * D, e0 + 2 * D, s, &g_self_k)));
  else
    DIF_TRY((gemm<T, T>(PK_GEMM_SELF_OUT, o, std::max(a, 8), lp.at<T>(lp.o_wo), std::max(a, 8), x, D,
                        M, D, a, dif::EPI_RESIDUAL, W.self_bo, mod + 2 * D, e0 + 2 * D, s)));

  // cross-attention to the text tokens
  {
    ProfScope ps(PK_NORM, s, 0, 2.0 * M * D * es);
    HIP_TRY(dif::launch_norm<T>(x, xn, M, D, 1, W.norm3_w, W.norm3_b, nullptr, nullptr, c.eps, s));
  }
  if (ac > 0) {
    T* cq = big;
    // With a text cache the step's K / V are the kept heads of the cached
    // all-head projections (the same values the projection below computes:
    // each output element's reduction is independent of which rows are kept).
    const bool cached = tk != nullptr;
    const int ldk = cached ? ac : 2 * ac;
    if (ix)
      DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_Q, xn, D, (const T*)W.cross_wq, D, cq, ac, M, ac, D,
                          dif::EPI_STORE, W.cross_bq, nullptr, nullptr, s, &g_cross_rows)));
    else
      DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_Q, xn, D, lp.at<T>(lp.o_wcq), D, cq, ac, M, ac, D,
                          dif::EPI_STORE, lp.at<float>(lp.o_bcq), nullptr, nullptr, s)));
    if (cached) {
      ProfScope ps(PK_GATHER, s, 0, 4.0 * Mc * ac * es);
      HIP_TRY(dif::launch_gather_cols16<T>(tk, D, ckv, ldk, Mc, ac, rc, s));
      HIP_TRY(dif::launch_gather_rows16<T>(tvt, (int64_t)D * wl.ldcvt, cvt, (int64_t)ac * wl.ldcvt,
                                           wl.ldcvt, ac, B, rc, s));
    } else if (ix) {
      dif::GemmGather g = g_cross_rows;
      g.nseg = 2;
      g.seg_b[0] = W.cross_wv;
      g.seg_bias[0] = W.cross_bv;
      DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_KV, ctx, D, (const T*)W.cross_wk, D, ckv, 2 * ac, Mc, ac, D,
                          dif::EPI_STORE, W.cross_bk, nullptr, nullptr, s, &g)));
    } else {
      DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_KV, ctx, D, lp.at<T>(lp.o_wckv), D, ckv, 2 * ac, Mc, 2 * ac, D,
                          dif::EPI_STORE, lp.at<float>(lp.o_bckv), nullptr, nullptr, s)));
    }
    {
      ProfScope ps(PK_QK_NORM, s, 0, 2.0 * (M + Mc) * ac * es);
      HIP_TRY(dif::launch_qk_norm<T>(cq, ac, M, ac, 1, 0, 0, ix ? W.cross_gq : lp.at<float>(lp.o_gcq),
                                     nullptr, inv_d, c.eps, nullptr, s, ix ? rc : nullptr, q_scale));
      HIP_TRY(dif::launch_qk_norm<T>(ckv, ldk, Mc, ac, 1, 0, 0,
                                     ix ? W.cross_gk : lp.at<float>(lp.o_gck), nullptr, inv_d, c.eps,
                                     nullptr, s, ix ? rc : nullptr));
    }
    if (!cached) {
      ProfScope ps(PK_TRANSPOSE, s, 0, 2.0 * Mc * ac * es);
      HIP_TRY(dif::launch_transpose_vt<T>(ckv + ac, 2 * ac, ac, B, Lc, cvt, wl.ldcvt, s));
    }
    DIF_TRY(attention<T>(PK_ATTN_CROSS, dh, cq, ac, ckv, ldk, cvt, wl.ldcvt, o, ac, B, L, Lc,
                         lp.info.cross_heads, s, true));
  }
  if (ix)
    DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_OUT, o, std::max(ac, 8), (const T*)W.cross_wo, D, x, D, M, D, ac,
                        dif::EPI_RESIDUAL, W.cross_bo, nullptr, nullptr, s, &g_cross_k)));
  else
    DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_OUT, o, std::max(ac, 8), lp.at<T>(lp.o_wco), std::max(ac, 8), x,
                        D, M, D, ac, dif::EPI_RESIDUAL, W.cross_bo, nullptr, nullptr, s)));

  // FFN: LN + AdaLN(shift2, scale2), GELU, gate2
  {
    ProfScope ps(PK_NORM, s, 0, 2.0 * M * D * es);
    HIP_TRY(dif::launch_norm<T>(x, xn, M, D, 0, mod + 3 * D, e0 + 3 * D, mod + 4 * D, e0 + 4 * D,
                                c.eps, s));
  }
  if (ix) {
    if (fp > 0)
      DIF_TRY((gemm<T, T>(PK_GEMM_FFN1, xn, D, (const T*)W.ffn_w1, D, big, fp, M, fp, D, dif::EPI_GELU,
                          W.ffn_b1, nullptr, nullptr, s, &g_ffn_rows)));
    DIF_TRY((gemm<T, T>(PK_GEMM_FFN2, big, std::max(fp, 8), (const T*)W.ffn_w2, c.ffn_dim, x, D, M, D,
                        fp, dif::EPI_RESIDUAL, W.ffn_b2, mod + 5 * D, e0 + 5 * D, s, &g_ffn_k)));
  } else {
    if (fp > 0)
      DIF_TRY((gemm<T, T>(PK_GEMM_FFN1, xn, D, lp.at<T>(lp.o_w1), D, big, fp, M, fp, D, dif::EPI_GELU,
                          lp.at<float>(lp.o_b1), nullptr, nullptr, s)));
    DIF_TRY((gemm<T, T>(PK_GEMM_FFN2, big, std::max(fp, 8), lp.at<T>(lp.o_w2), std::max(fp, 8), x, D,
                        M, D, fp, dif::EPI_RESIDUAL, W.ffn_b2, mod + 5 * D, e0 + 5 * D, s)));
  }
  return DIF_OK;
}

template <typename T>
dif_status time_embed_impl(const dif_model* m, float t, float* e, float* e0, char* ws,
                           const WsLayout& wl, hipStream_t s) {
  const dif_config& c = m->cfg;
  const int D = c.dim, Fq = c.freq_dim;
  float* emb = reinterpret_cast<float*>(ws + wl.emb);
  float* t1 = reinterpret_cast<float*>(ws + wl.t1);
  float* t2 = reinterpret_cast<float*>(ws + wl.t2);
  ProfScope ps(PK_TIME_EMBED, s, 2.0 * D * (Fq + D + 6.0 * D),
               sizeof(T) * (double)D * (Fq + D + 6.0 * D));
  HIP_TRY(dif::launch_sinusoid(t, Fq, emb, s));
  HIP_TRY(dif::launch_gemv<T>((const T*)m->w.t_w1, emb, m->w.t_b1, t1, D, Fq, s));
  HIP_TRY(dif::launch_silu(t1, t2, D, s));
  HIP_TRY(dif::launch_gemv<T>((const T*)m->w.t_w2, t2, m->w.t_b2, e, D, D, s));
  HIP_TRY(dif::launch_silu(e, t1, D, s));
  HIP_TRY(dif::launch_gemv<T>((const T*)m->w.t_w3, t1, m->w.t_b3, e0, 6 * D, D, s));
  return DIF_OK;
}

// All layers' text projections for context ctx [B, Lc, D].
template <typename T>
dif_status text_cache_impl(const dif_model* m, const T* ctx, int B, int Lc, char* cache,
                           const TextLayout& tl, hipStream_t s) {
  const dif_config& c = m->cfg;
  const int D = c.dim, Mc = B * Lc;
  T* stage = reinterpret_cast<T*>(cache + tl.stage);
  for (int l = 0; l < c.n_layers; ++l) {
    const dif_layer_weights& W = m->layers[l];
    T* k = reinterpret_cast<T*>(cache + tl.k(l));
    T* vt = reinterpret_cast<T*>(cache + tl.vt(l));
    DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_KV, ctx, D, (const T*)W.cross_wk, D, k, D, Mc, D, D,
                        dif::EPI_STORE, W.cross_bk, nullptr, nullptr, s)));
    DIF_TRY((gemm<T, T>(PK_GEMM_CROSS_KV, ctx, D, (const T*)W.cross_wv, D, stage, D, Mc, D, D,
                        dif::EPI_STORE, W.cross_bv, nullptr, nullptr, s)));
    ProfScope ps(PK_TRANSPOSE, s, 0, 2.0 * Mc * D * sizeof(T));
    HIP_TRY(dif::launch_transpose_vt<T>(stage, D, D, B, Lc, vt, tl.ldcvt, s));
  }
  return DIF_OK;
}

template <typename T>
dif_status step_impl(const dif_plan* plan, const float* z, float t, const T* ctx, int B, int L,
                     int Lc, float* v, char* ws, const WsLayout& wl, hipStream_t s,
                     const char* cache = nullptr, const TextLayout* tl = nullptr) {
  const dif_model* m = plan->model;
  const dif_config& c = m->cfg;
  const int D = c.dim, Cp = c.patch_dim, M = B * L;
  float* e = reinterpret_cast<float*>(ws + wl.e);
  float* e0 = reinterpret_cast<float*>(ws + wl.e0);
  T* x = reinterpret_cast<T*>(ws + wl.x);
  T* xn = reinterpret_cast<T*>(ws + wl.xn);
  DIF_TRY(time_embed_impl<T>(m, t, e, e0, ws, wl, s));
  const T* zin;
  if constexpr (sizeof(T) == 4) {
    zin = reinterpret_cast<const T*>(z);
  } else {
    T* zc = reinterpret_cast<T*>(ws + wl.zc);
    ProfScope ps(PK_ELEMENTWISE, s, 0, 6.0 * M * Cp);
    HIP_TRY(dif::launch_cast<T>(z, zc, (int64_t)M * Cp, s));
    zin = zc;
  }
  DIF_TRY((gemm<T, T>(PK_GEMM_IO, zin, Cp, (const T*)m->w.patch_w, Cp, x, D, M, D, Cp,
                      dif::EPI_STORE, m->w.patch_b, nullptr, nullptr, s)));
  for (int l = 0; l < c.n_layers; ++l) {
    const T* tk = cache ? reinterpret_cast<const T*>(cache + tl->k(l)) : nullptr;
    const T* tvt = cache ? reinterpret_cast<const T*>(cache + tl->vt(l)) : nullptr;
    DIF_TRY(block_impl<T>(plan, l, x, ctx, e0, B, L, Lc, ws, wl, s, tk, tvt));
  }
  {
    ProfScope ps(PK_NORM, s, 0, 2.0 * M * D * sizeof(T));
    HIP_TRY(dif::launch_norm<T>(x, xn, M, D, 0, m->w.head_mod, e, m->w.head_mod + D, e, c.eps, s));
  }
  DIF_TRY((gemm<T, float>(PK_GEMM_IO, xn, D, (const T*)m->w.head_w, D, v, Cp, M, Cp, D,
                          dif::EPI_STORE, m->w.head_b, nullptr, nullptr, s)));
  return DIF_OK;
}

dif_status check_run(const dif_plan* plan, int B, int L, int Lc) {
  if (!plan || !plan->model) return fail(DIF_E_ARG, "plan is null");
  const dif_config& c = plan->model->cfg;
  if (B <= 0) return fail(DIF_E_SHAPE, "B must be >= 1");
  if ((int64_t)L != (int64_t)c.grid_f * c.grid_h * c.grid_w)
    return fail(DIF_E_SHAPE, "L = %d does not match the token grid %dx%dx%d", L, c.grid_f, c.grid_h,
                c.grid_w);
  if (Lc < 1 || Lc > c.max_text_len) return fail(DIF_E_SHAPE, "Lc = %d outside [1, %d]", Lc, c.max_text_len);
  if ((int64_t)B * L > (1 << 30) / 8) return fail(DIF_E_SHAPE, "B * L too large");
  return DIF_OK;
}

bool is_gfx950() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return false;
  return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
}

}  // namespace

namespace {

// Shared by the calls with a context (cache == null) and with a text cache
// (ctx unused).
dif_status block_call(const dif_plan* plan, int32_t layer, void* x, const void* ctx,
                      const void* cache, size_t cache_bytes, const float* e0, int32_t B, int32_t L,
                      int32_t Lc, void* ws, size_t ws_bytes, dif_stream stream) {
  DIF_TRY(check_run(plan, B, L, Lc));
  const dif_config& c = plan->model->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(DIF_E_ARG, "layer %d out of range", layer);
  if (!x || (!ctx && !cache) || !e0) return fail(DIF_E_ARG, "null tensor argument");
  const TextLayout tl = text_layout(c, B, Lc);
  if (cache) DIF_TRY(check_cache(tl, cache, cache_bytes));
  const WsLayout wl = ws_layout(c, B, L, Lc);
  DIF_TRY(check_ws(wl, ws, ws_bytes));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const char* cb = static_cast<const char*>(cache);
  if (c.dtype == DIF_BF16)
    return block_impl<bf16>(plan, layer, (bf16*)x, (const bf16*)ctx, e0, B, L, Lc, w, wl, s,
                            cb ? (const bf16*)(cb + tl.k(layer)) : nullptr,
                            cb ? (const bf16*)(cb + tl.vt(layer)) : nullptr);
  return block_impl<float>(plan, layer, (float*)x, (const float*)ctx, e0, B, L, Lc, w, wl, s,
                           cb ? (const float*)(cb + tl.k(layer)) : nullptr,
                           cb ? (const float*)(cb + tl.vt(layer)) : nullptr);
}

dif_status step_call(const dif_plan* plan, const float* z, float t, const void* ctx,
                     const void* cache, size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                     float* v_out, void* ws, size_t ws_bytes, dif_stream stream) {
  DIF_TRY(check_run(plan, B, L, Lc));
  const dif_config& c = plan->model->cfg;
  if (!z || (!ctx && !cache) || !v_out) return fail(DIF_E_ARG, "null tensor argument");
  if (!std::isfinite(t)) return fail(DIF_E_ARG, "timestep is not finite");
  if (!(plan->flags & DIF_PLAN_ANY_T) && t != plan->t_s)
    return fail(DIF_E_ARG, "timestep %g differs from the plan's t_s = %g (step %d)", (double)t,
                (double)plan->t_s, plan->step);
  const TextLayout tl = text_layout(c, B, Lc);
  if (cache) DIF_TRY(check_cache(tl, cache, cache_bytes));
  const WsLayout wl = ws_layout(c, B, L, Lc);
  DIF_TRY(check_ws(wl, ws, ws_bytes));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const char* cb = static_cast<const char*>(cache);
  return c.dtype == DIF_BF16
             ? step_impl<bf16>(plan, z, t, (const bf16*)ctx, B, L, Lc, v_out, w, wl, s, cb, &tl)
             : step_impl<float>(plan, z, t, (const float*)ctx, B, L, Lc, v_out, w, wl, s, cb, &tl);
}

dif_status rollout_call(const dif_plan* const* plans, const float* timesteps, int32_t n_steps,
                        int32_t sampler, float* z, const float* const* eps, const void* ctx,
                        const void* cache, size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                        float* v_scratch, void* ws, size_t ws_bytes, dif_stream stream) {
  if (!plans || !timesteps || !z || (!ctx && !cache) || !v_scratch) return fail(DIF_E_ARG, "null argument");
  if (n_steps < 1) return fail(DIF_E_ARG, "n_steps must be >= 1");
  if (sampler != DIF_SAMPLER_EULER && sampler != DIF_SAMPLER_RENOISE)
    return fail(DIF_E_ARG, "unknown sampler %d", sampler);
  for (int i = 0; i < n_steps; ++i) {
    if (!plans[i]) return fail(DIF_E_ARG, "plan %d is null", i);
    if (plans[i]->model != plans[0]->model) return fail(DIF_E_ARG, "plans of different models");
    if (!std::isfinite(timesteps[i])) return fail(DIF_E_ARG, "timestep %d is not finite", i);
    if (!(plans[i]->flags & DIF_PLAN_ANY_T) && timesteps[i] != plans[i]->t_s)
      return fail(DIF_E_ARG, "timestep %d = %g differs from its plan's t_s = %g", i,
                  (double)timesteps[i], (double)plans[i]->t_s);
    if (sampler == DIF_SAMPLER_RENOISE && i + 1 < n_steps && (!eps || !eps[i]))
      return fail(DIF_E_ARG, "re-noise sampler needs eps[%d]", i);
  }
  const int64_t n = (int64_t)B * L * plans[0]->model->cfg.patch_dim;
  for (int i = 0; i < n_steps; ++i) {
    DIF_TRY(step_call(plans[i], z, timesteps[i], ctx, cache, cache_bytes, B, L, Lc, v_scratch, ws,
                      ws_bytes, stream));
    const float sf = timesteps[i] / 1000.f;
    const float st = i + 1 < n_steps ? timesteps[i + 1] / 1000.f : 0.f;
    if (sampler == DIF_SAMPLER_EULER)
      DIF_TRY(dif_euler(z, v_scratch, sf, st, n, stream));
    else
      DIF_TRY(dif_renoise(z, v_scratch, sf, st, i + 1 < n_steps ? eps[i] : nullptr, n, stream));
  }
  return DIF_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* dif_last_error(void) { return g_err.c_str(); }

dif_status dif_validate_config(const dif_config* cfg) {
  GUARD_BEGIN
  return check_config(cfg);
  GUARD_END
}

dif_status dif_validate_masks(const dif_config* cfg, const dif_step_masks* masks) {
  GUARD_BEGIN
  DIF_TRY(check_config(cfg));
  return check_masks(cfg, masks);
  GUARD_END
}

dif_status dif_model_create(const dif_config* cfg, const dif_weights* w, dif_model** out) {
  GUARD_BEGIN
  if (!out) return fail(DIF_E_ARG, "out is null");
  *out = nullptr;
  DIF_TRY(check_config(cfg));
  if (!w || !w->layers) return fail(DIF_E_ARG, "weights are null");
  const void* g[] = {w->patch_w, w->patch_b, w->t_w1, w->t_b1, w->t_w2, w->t_b2, w->t_w3,
                     w->t_b3, w->head_mod, w->head_w, w->head_b};
  for (const void* p : g)
    if (!p) return fail(DIF_E_ARG, "a global weight pointer is null");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const dif_layer_weights& L = w->layers[l];
    const void* ps[] = {L.mod, L.self_wq, L.self_wk, L.self_wv, L.self_wo, L.self_bq, L.self_bk,
                        L.self_bv, L.self_bo, L.self_gq, L.self_gk, L.norm3_w, L.norm3_b,
                        L.cross_wq, L.cross_wk, L.cross_wv, L.cross_wo, L.cross_bq, L.cross_bk,
                        L.cross_bv, L.cross_bo, L.cross_gq, L.cross_gk, L.ffn_w1, L.ffn_b1,
                        L.ffn_w2, L.ffn_b2};
    for (const void* p : ps)
      if (!p) return fail(DIF_E_ARG, "layer %d has a null weight pointer", l);
  }
  if (!is_gfx950()) return fail(DIF_E_UNSUPPORTED, "current HIP device is not gfx950");
  int dev = 0, ncu = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
  dif_model* m = new dif_model();
  m->cfg = *cfg;
  m->ncu = ncu;
  m->w = *w;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->w.layers = nullptr;
  *out = m;
  return DIF_OK;
  GUARD_END
}

dif_status dif_model_destroy(dif_model* model) {
  delete model;
  return DIF_OK;
}

dif_status dif_plan_bytes_ex(const dif_model* model, const dif_step_masks* masks, int32_t kind,
                            size_t* bytes) {
  GUARD_BEGIN
  if (!model || !bytes) return fail(DIF_E_ARG, "null argument");
  DIF_TRY(check_plan_kind(&model->cfg, kind));
  DIF_TRY(check_masks(&model->cfg, masks));
  *bytes = build_layout(model, masks, kind == DIF_PLAN_INDEXED).total;
  return DIF_OK;
  GUARD_END
}

dif_status dif_plan_bytes(const dif_model* model, const dif_step_masks* masks, size_t* bytes) {
  return dif_plan_bytes_ex(model, masks, DIF_PLAN_COMPACT, bytes);
}

dif_status dif_plan_step(const dif_model* model, int32_t step, float t_s,
                         const dif_step_masks* masks, void* plan_mem, size_t plan_bytes,
                         dif_stream stream, dif_plan** out) {
  return dif_plan_step_ex(model, step, t_s, masks, DIF_PLAN_COMPACT, 0, plan_mem, plan_bytes,
                          stream, out);
}

dif_status dif_plan_step_ex(const dif_model* model, int32_t step, float t_s,
                            const dif_step_masks* masks, int32_t kind, int32_t flags,
                            void* plan_mem, size_t plan_bytes, dif_stream stream, dif_plan** out) {
  GUARD_BEGIN
  if (!model || !out) return fail(DIF_E_ARG, "null argument");
  *out = nullptr;
  if (step < 0 || step >= 4096) return fail(DIF_E_ARG, "step %d out of range", step);
  if (flags & ~DIF_PLAN_ANY_T) return fail(DIF_E_ARG, "unknown plan flags 0x%x", flags);
  if (!(flags & DIF_PLAN_ANY_T) && !std::isfinite(t_s))
    return fail(DIF_E_ARG, "t_s is not finite (pass DIF_PLAN_ANY_T for an unbound plan)");
  DIF_TRY(check_plan_kind(&model->cfg, kind));
  DIF_TRY(check_masks(&model->cfg, masks));
  Layout lay = build_layout(model, masks, kind == DIF_PLAN_INDEXED);
  if (!plan_mem) return fail(DIF_E_WORKSPACE, "plan memory is null");
  if (reinterpret_cast<uintptr_t>(plan_mem) % 256) return fail(DIF_E_WORKSPACE, "plan memory not 256-byte aligned");
  if (plan_bytes < lay.total)
    return fail(DIF_E_WORKSPACE, "plan memory %zu bytes < required %zu", plan_bytes, lay.total);
  const dif_config& c = model->cfg;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  dif_plan* p = new dif_plan();
  p->model = model;
  p->step = step;
  p->t_s = t_s;
  p->flags = flags;
  p->lay = std::move(lay);
  p->mem = static_cast<char*>(plan_mem);
  p->bytes = plan_bytes;
  for (auto& lp : p->lay.layers) lp.base = p->mem;

  // RoPE table: (cos, sin) of pos * theta^(-2j/d_axis) per axis, computed in double
  int jt, jh, jw;
  rope_pairs(c.head_dim, &jt, &jh, &jw);
  p->host_rope.resize(p->lay.n_rope * 2);
  size_t k = 0;
  const int np[3] = {jt, jh, jw}, gp[3] = {c.grid_f, c.grid_h, c.grid_w};
  for (int ax = 0; ax < 3; ++ax)
    for (int pos = 0; pos < gp[ax]; ++pos)
      for (int j = 0; j < np[ax]; ++j) {
        const double ang = pos * std::pow((double)c.rope_theta, -2.0 * j / (2.0 * np[ax]));
        p->host_rope[k++] = (float)std::cos(ang);
        p->host_rope[k++] = (float)std::sin(ang);
      }
  p->rope = dif::RopeDesc{reinterpret_cast<const float*>(p->mem + p->lay.o_rope), 0, c.grid_f, c.grid_h,
                          c.grid_w, jt, jh, jw, c.head_dim};
  auto cleanup = [&](dif_status st) {
    delete p;
    return st;
  };
  if (hipMemcpyAsync(p->mem + p->lay.o_rope, p->host_rope.data(), p->host_rope.size() * sizeof(float),
                     hipMemcpyHostToDevice, s) != hipSuccess)
    return cleanup(fail(DIF_E_HIP, "rope table upload failed"));
  if (!p->lay.host_idx.empty() &&
      hipMemcpyAsync(p->mem + p->lay.o_idx, p->lay.host_idx.data(),
                     p->lay.host_idx.size() * sizeof(int32_t), hipMemcpyHostToDevice, s) != hipSuccess)
    return cleanup(fail(DIF_E_HIP, "index table upload failed"));
  for (int l = 0; l < c.n_layers && !p->lay.indexed; ++l) {
    const LayerPlan& lp = p->lay.layers[l];
    if (!lp.info.block_keep) continue;
    const dif_status st = c.dtype == DIF_BF16 ? gather_layer<bf16>(model, l, lp, s)
                                              : gather_layer<float>(model, l, lp, s);
    if (st != DIF_OK) return cleanup(st);
  }
  *out = p;
  return DIF_OK;
  GUARD_END
}

dif_status dif_plan_destroy(dif_plan* plan) {
  delete plan;
  return DIF_OK;
}

dif_status dif_plan_timestep(const dif_plan* plan, float* t_s, int32_t* flags) {
  if (!plan || !t_s || !flags) return fail(DIF_E_ARG, "null argument");
  *t_s = plan->t_s;
  *flags = plan->flags;
  return DIF_OK;
}

dif_status dif_plan_layer_info(const dif_plan* plan, int32_t layer, dif_layer_info* out) {
  if (!plan || !out) return fail(DIF_E_ARG, "null argument");
  if (layer < 0 || layer >= (int)plan->lay.layers.size()) return fail(DIF_E_ARG, "layer out of range");
  *out = plan->lay.layers[layer].info;
  return DIF_OK;
}

dif_status dif_workspace_bytes(const dif_model* model, int32_t B, int32_t L, int32_t Lc, size_t* bytes) {
  GUARD_BEGIN
  if (!model || !bytes) return fail(DIF_E_ARG, "null argument");
  if (B <= 0 || L <= 0 || Lc <= 0) return fail(DIF_E_SHAPE, "B, L, Lc must be >= 1");
  *bytes = ws_layout(model->cfg, B, L, Lc).total;
  return DIF_OK;
  GUARD_END
}

dif_status dif_time_embed(const dif_model* model, float t, float* e_out, float* e0_out, void* ws,
                          size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!model || !e_out || !e0_out) return fail(DIF_E_ARG, "null argument");
  const WsLayout wl = ws_layout(model->cfg, 1, 1, 1);
  DIF_TRY(check_ws(wl, ws, ws_bytes));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  return model->cfg.dtype == DIF_BF16
             ? time_embed_impl<bf16>(model, t, e_out, e0_out, static_cast<char*>(ws), wl, s)
             : time_embed_impl<float>(model, t, e_out, e0_out, static_cast<char*>(ws), wl, s);
  GUARD_END
}


dif_status dif_block_forward(const dif_plan* plan, int32_t layer, void* x, const void* ctx,
                             const float* e0, int32_t B, int32_t L, int32_t Lc, void* ws,
                             size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!ctx) return fail(DIF_E_ARG, "null tensor argument");
  return block_call(plan, layer, x, ctx, nullptr, 0, e0, B, L, Lc, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_block_forward_cached(const dif_plan* plan, int32_t layer, void* x, const void* cache,
                                    size_t cache_bytes, const float* e0, int32_t B, int32_t L,
                                    int32_t Lc, void* ws, size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!cache) return fail(DIF_E_ARG, "text cache is null");
  return block_call(plan, layer, x, nullptr, cache, cache_bytes, e0, B, L, Lc, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_step_forward(const dif_plan* plan, const float* z, float t, const void* ctx, int32_t B,
                            int32_t L, int32_t Lc, float* v_out, void* ws, size_t ws_bytes,
                            dif_stream stream) {
  GUARD_BEGIN
  if (!ctx) return fail(DIF_E_ARG, "null tensor argument");
  return step_call(plan, z, t, ctx, nullptr, 0, B, L, Lc, v_out, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_step_forward_cached(const dif_plan* plan, const float* z, float t, const void* cache,
                                   size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                                   float* v_out, void* ws, size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!cache) return fail(DIF_E_ARG, "text cache is null");
  return step_call(plan, z, t, nullptr, cache, cache_bytes, B, L, Lc, v_out, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_text_cache_bytes(const dif_model* model, int32_t B, int32_t Lc, size_t* bytes) {
  GUARD_BEGIN
  if (!model || !bytes) return fail(DIF_E_ARG, "null argument");
  DIF_TRY(check_text(model->cfg, B, Lc));
  *bytes = text_layout(model->cfg, B, Lc).total;
  return DIF_OK;
  GUARD_END
}

dif_status dif_text_cache_build(const dif_model* model, const void* ctx, int32_t B, int32_t Lc,
                                void* cache, size_t cache_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!model || !ctx) return fail(DIF_E_ARG, "null argument");
  const dif_config& c = model->cfg;
  DIF_TRY(check_text(c, B, Lc));
  const TextLayout tl = text_layout(c, B, Lc);
  DIF_TRY(check_cache(tl, cache, cache_bytes));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* cb = static_cast<char*>(cache);
  return c.dtype == DIF_BF16 ? text_cache_impl<bf16>(model, (const bf16*)ctx, B, Lc, cb, tl, s)
                             : text_cache_impl<float>(model, (const float*)ctx, B, Lc, cb, tl, s);
  GUARD_END
}

dif_status dif_euler(float* z, const float* v, float sigma_from, float sigma_to, int64_t n,
                     dif_stream stream) {
  GUARD_BEGIN
  if (!z || !v) return fail(DIF_E_ARG, "null argument");
  if (n < 0) return fail(DIF_E_SHAPE, "n < 0");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  ProfScope ps(PK_ELEMENTWISE, s, 2.0 * n, 12.0 * n);
  HIP_TRY(dif::launch_euler(z, v, sigma_to - sigma_from, n, s));
  return DIF_OK;
  GUARD_END
}

dif_status dif_renoise(float* z, const float* v, float sigma_from, float sigma_to, const float* eps,
                       int64_t n, dif_stream stream) {
  GUARD_BEGIN
  if (!z || !v) return fail(DIF_E_ARG, "null argument");
  if (n < 0) return fail(DIF_E_SHAPE, "n < 0");
  if (!std::isfinite(sigma_from) || !std::isfinite(sigma_to) || sigma_to < 0.f || sigma_to > 1.f)
    return fail(DIF_E_ARG, "sigma_from must be finite and 0 <= sigma_to <= 1");
  if (sigma_to != 0.f && !eps) return fail(DIF_E_ARG, "eps is null but sigma_to = %g", sigma_to);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  ProfScope ps(PK_ELEMENTWISE, s, 4.0 * n, (sigma_to != 0.f ? 16.0 : 12.0) * n);
  HIP_TRY(dif::launch_renoise(z, v, sigma_from, sigma_to, sigma_to != 0.f ? eps : nullptr, n, s));
  return DIF_OK;
  GUARD_END
}


dif_status dif_rollout(const dif_plan* const* plans, const float* timesteps, int32_t n_steps,
                       int32_t sampler, float* z, const float* const* eps, const void* ctx,
                       int32_t B, int32_t L, int32_t Lc, float* v_scratch, void* ws,
                       size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!ctx) return fail(DIF_E_ARG, "null argument");
  return rollout_call(plans, timesteps, n_steps, sampler, z, eps, ctx, nullptr, 0, B, L, Lc,
                      v_scratch, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_rollout_cached(const dif_plan* const* plans, const float* timesteps, int32_t n_steps,
                              int32_t sampler, float* z, const float* const* eps, const void* cache,
                              size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                              float* v_scratch, void* ws, size_t ws_bytes, dif_stream stream) {
  GUARD_BEGIN
  if (!cache) return fail(DIF_E_ARG, "text cache is null");
  return rollout_call(plans, timesteps, n_steps, sampler, z, eps, nullptr, cache, cache_bytes, B, L,
                      Lc, v_scratch, ws, ws_bytes, stream);
  GUARD_END
}

dif_status dif_hard_gates(const dif_config* cfg, int32_t chunk, const float* m_block,
                          const float* m_self, const float* m_cross, const float* m_ffn,
                          uint8_t* block_keep, uint8_t* self_head_keep, uint8_t* cross_head_keep,
                          uint8_t* ffn_keep) {
  GUARD_BEGIN
  DIF_TRY(check_config(cfg));
  if (!m_block || !m_self || !m_cross || !m_ffn || !block_keep || !self_head_keep ||
      !cross_head_keep || !ffn_keep)
    return fail(DIF_E_ARG, "null argument");
  const int N = cfg->n_layers, H = cfg->n_heads, dh = cfg->head_dim, F = cfg->ffn_dim;
  if (chunk < 1 || F % chunk != 0)
    return fail(DIF_E_SHAPE, "ffn_dim %d is not a multiple of the chunk %d", F, chunk);
  const int nc = F / chunk;
  for (int l = 0; l < N; ++l) {
    block_keep[l] = m_block[l] > 0.f ? 1 : 0;
    const float* ms[2] = {m_self + (size_t)l * H * dh, m_cross + (size_t)l * H * dh};
    uint8_t* ks[2] = {self_head_keep + (size_t)l * H, cross_head_keep + (size_t)l * H};
    for (int a = 0; a < 2; ++a)
      for (int h = 0; h < H; ++h) {
        double sum = 0.0;   // mean > 0  <=>  sum > 0
        for (int d = 0; d < dh; ++d) sum += (double)ms[a][h * dh + d];
        ks[a][h] = sum > 0.0 ? 1 : 0;
      }
    for (int c = 0; c < nc; ++c) {
      const uint8_t g = m_ffn[(size_t)l * nc + c] > 0.f ? 1 : 0;
      std::memset(ffn_keep + (size_t)l * F + (size_t)c * chunk, g, chunk);
    }
  }
  return DIF_OK;
  GUARD_END
}

dif_status dif_ffn_reorder(const dif_model* model, int32_t layer, void* w1_out, float* b1_out,
                           void* w2_out, int32_t* perm_out, void* scratch, size_t scratch_bytes,
                           dif_stream stream) {
  GUARD_BEGIN
  if (!model || !w1_out || !b1_out || !w2_out || !perm_out || !scratch)
    return fail(DIF_E_ARG, "null argument");
  const dif_config& c = model->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(DIF_E_ARG, "layer %d out of range", layer);
  const int D = c.dim, F = c.ffn_dim;
  if (scratch_bytes < (size_t)F * (sizeof(double) + sizeof(int32_t)))
    return fail(DIF_E_WORKSPACE, "scratch %zu bytes < %zu", scratch_bytes,
                (size_t)F * (sizeof(double) + sizeof(int32_t)));
  if (reinterpret_cast<uintptr_t>(scratch) % 8) return fail(DIF_E_WORKSPACE, "scratch not 8-byte aligned");
  const dif_layer_weights& W = model->layers[layer];
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  double* norms = static_cast<double*>(scratch);
  int32_t* dperm = reinterpret_cast<int32_t*>(norms + F);
  if (c.dtype == DIF_BF16)
    HIP_TRY(dif::launch_ffn_norms<bf16>((const bf16*)W.ffn_w1, W.ffn_b1, (const bf16*)W.ffn_w2, D, F,
                                        norms, s));
  else
    HIP_TRY(dif::launch_ffn_norms<float>((const float*)W.ffn_w1, W.ffn_b1, (const float*)W.ffn_w2, D,
                                         F, norms, s));
  std::vector<double> hn(F);
  HIP_TRY(hipMemcpyAsync(hn.data(), norms, F * sizeof(double), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  std::vector<int32_t> perm(F);
  for (int j = 0; j < F; ++j) perm[j] = j;
  std::stable_sort(perm.begin(), perm.end(), [&](int32_t a, int32_t b) { return hn[a] > hn[b]; });
  std::memcpy(perm_out, perm.data(), F * sizeof(int32_t));
  HIP_TRY(hipMemcpyAsync(dperm, perm.data(), F * sizeof(int32_t), hipMemcpyHostToDevice, s));
  if (c.dtype == DIF_BF16) {
    HIP_TRY(dif::launch_gather<bf16>((const bf16*)W.ffn_w1, D, (bf16*)w1_out, D, F, D, dperm, nullptr, s));
    HIP_TRY(dif::launch_gather<bf16>((const bf16*)W.ffn_w2, F, (bf16*)w2_out, F, D, F, nullptr, dperm, s));
  } else {
    HIP_TRY(dif::launch_gather<float>((const float*)W.ffn_w1, D, (float*)w1_out, D, F, D, dperm, nullptr, s));
    HIP_TRY(dif::launch_gather<float>((const float*)W.ffn_w2, F, (float*)w2_out, F, D, F, nullptr, dperm, s));
  }
  HIP_TRY(dif::launch_gather<float>(W.ffn_b1, 1, b1_out, 1, F, 1, dperm, nullptr, s));
  HIP_TRY(hipStreamSynchronize(s));   // the host permutation buffer is released on return
  return DIF_OK;
  GUARD_END
}

dif_status dif_gemm(int32_t dtype, int32_t out_dtype, const void* A, int64_t lda, const void* B,
                    int64_t ldb, void* C, int64_t ldc, int32_t M, int32_t N, int32_t K,
                    int32_t epilogue, const float* bias, const float* gate0, const float* gate1,
                    dif_stream stream) {
  GUARD_BEGIN
  if (dtype != DIF_BF16 && dtype != DIF_F32) return fail(DIF_E_ARG, "bad dtype");
  if (out_dtype != dtype && out_dtype != DIF_F32) return fail(DIF_E_ARG, "bad out_dtype");
  if (epilogue < 0 || epilogue > 2) return fail(DIF_E_ARG, "bad epilogue");
  if (M < 0 || N < 0 || K < 0) return fail(DIF_E_SHAPE, "negative size");
  const int64_t es = esize(dtype), kt = 128 / es;
  if (K % kt) return fail(DIF_E_SHAPE, "K = %d not a multiple of %lld", K, (long long)kt);
  if (M == 0 || N == 0) return DIF_OK;
  if (!C) return fail(DIF_E_ARG, "null output");
  if (ldc < N) return fail(DIF_E_SHAPE, "ldc < N");
  // the kernels address 256-row blocks through 32-bit buffer descriptors
  const int64_t oes = esize(out_dtype), kBlock = 256, kSpan = int64_t(1) << 31;
  if (kBlock * ldc * oes >= kSpan || (K > 0 && kBlock * std::max(lda, ldb) * es >= kSpan))
    return fail(DIF_E_SHAPE, "256 rows of a matrix span 2 GiB or more");
  if (K > 0) {  // A and B are read only when K > 0
    if (!A || !B) return fail(DIF_E_ARG, "null operand");
    if (lda < K || ldb < K) return fail(DIF_E_SHAPE, "leading dimension too small");
    if ((lda * es) % 16 || (ldb * es) % 16)
      return fail(DIF_E_SHAPE, "lda and ldb must be 16-byte multiples");
    if ((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(B)) % 16)
      return fail(DIF_E_ARG, "A and B must be 16-byte aligned");
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (dtype == DIF_BF16 && out_dtype == DIF_BF16)
    return gemm<bf16, bf16>(PK_GEMM_IO, (const bf16*)A, lda, (const bf16*)B, ldb, (bf16*)C, ldc, M,
                            N, K, epilogue, bias, gate0, gate1, s);
  if (dtype == DIF_BF16)
    return gemm<bf16, float>(PK_GEMM_IO, (const bf16*)A, lda, (const bf16*)B, ldb, (float*)C, ldc,
                             M, N, K, epilogue, bias, gate0, gate1, s);
  return gemm<float, float>(PK_GEMM_IO, (const float*)A, lda, (const float*)B, ldb, (float*)C, ldc,
                            M, N, K, epilogue, bias, gate0, gate1, s);
  GUARD_END
}

}  // extern "C"

namespace {

// Shared by dif_attention and dif_attention_ex: validation, then the launch
// (split_ws null: unsplit).
dif_status attention_call(int32_t dtype, int32_t head_dim, int32_t flags, const void* Q,
                          int64_t ldq, const void* K, int64_t ldk, const void* Vt, int64_t ldvt,
                          void* O, int64_t ldo, int32_t B, int32_t Lq, int32_t Lk,
                          int32_t n_heads, float* split_ws, size_t split_ws_bytes,
                          dif_stream stream) {
  if (dtype != DIF_BF16 && dtype != DIF_F32) return fail(DIF_E_ARG, "bad dtype");
  if (head_dim != 64 && head_dim != 128) return fail(DIF_E_UNSUPPORTED, "head_dim %d", head_dim);
  if (flags & ~DIF_ATTN_Q_PRESCALED) return fail(DIF_E_ARG, "unknown attention flags 0x%x", flags);
  if (B < 0 || Lq < 0 || n_heads < 0) return fail(DIF_E_SHAPE, "negative size");
  if (Lk < 1) return fail(DIF_E_SHAPE, "Lk must be >= 1");
  if (split_ws) {
    if (reinterpret_cast<uintptr_t>(split_ws) % 256)
      return fail(DIF_E_WORKSPACE, "split workspace not 256-byte aligned");
    if (split_ws_bytes < dif::attention_split_bytes(head_dim))
      return fail(DIF_E_WORKSPACE, "split workspace %zu bytes < required %zu", split_ws_bytes,
                  dif::attention_split_bytes(head_dim));
  }
  if (B == 0 || Lq == 0 || n_heads == 0) return DIF_OK;
  if (!Q || !K || !Vt || !O) return fail(DIF_E_ARG, "null tensor");
  const int64_t es = esize(dtype);
  const int64_t w = (int64_t)n_heads * head_dim;
  if (ldq < w || ldk < w || ldo < w || ldvt < Lk) return fail(DIF_E_SHAPE, "leading dimension too small");
  if ((ldq * es) % 16 || (ldk * es) % 16 || (ldo * es) % 16 || (ldvt * es) % 16)
    return fail(DIF_E_SHAPE, "leading dimensions must be 16-byte multiples");
  if ((reinterpret_cast<uintptr_t>(Q) | reinterpret_cast<uintptr_t>(K) |
       reinterpret_cast<uintptr_t>(Vt) | reinterpret_cast<uintptr_t>(O)) % 16)
    return fail(DIF_E_ARG, "tensors must be 16-byte aligned");
  int ncu = 0;
  if (split_ws) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    HIP_TRY(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
  }
  const bool pre = (flags & DIF_ATTN_Q_PRESCALED) != 0;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (dtype == DIF_BF16)
    return attention<bf16>(PK_ATTN_SELF, head_dim, (const bf16*)Q, ldq, (const bf16*)K, ldk,
                           (const bf16*)Vt, ldvt, (bf16*)O, ldo, B, Lq, Lk, n_heads, s, pre,
                           split_ws, ncu);
  return attention<float>(PK_ATTN_SELF, head_dim, (const float*)Q, ldq, (const float*)K, ldk,
                          (const float*)Vt, ldvt, (float*)O, ldo, B, Lq, Lk, n_heads, s, pre,
                          split_ws, ncu);
}

}  // namespace

extern "C" {

dif_status dif_attention(int32_t dtype, int32_t head_dim, const void* Q, int64_t ldq, const void* K,
                         int64_t ldk, const void* Vt, int64_t ldvt, void* O, int64_t ldo, int32_t B,
                         int32_t Lq, int32_t Lk, int32_t n_heads, dif_stream stream) {
  GUARD_BEGIN
  return attention_call(dtype, head_dim, 0, Q, ldq, K, ldk, Vt, ldvt, O, ldo, B, Lq, Lk, n_heads,
                        nullptr, 0, stream);
  GUARD_END
}

dif_status dif_attention_split_bytes(int32_t head_dim, size_t* bytes) {
  if (!bytes) return fail(DIF_E_ARG, "null argument");
  if (head_dim != 64 && head_dim != 128) return fail(DIF_E_UNSUPPORTED, "head_dim %d", head_dim);
  *bytes = dif::attention_split_bytes(head_dim);
  return DIF_OK;
}

dif_status dif_attention_ex(int32_t dtype, int32_t head_dim, int32_t flags, const void* Q,
                            int64_t ldq, const void* K, int64_t ldk, const void* Vt, int64_t ldvt,
                            void* O, int64_t ldo, int32_t B, int32_t Lq, int32_t Lk,
                            int32_t n_heads, void* split_ws, size_t split_ws_bytes,
                            dif_stream stream) {
  GUARD_BEGIN
  return attention_call(dtype, head_dim, flags, Q, ldq, K, ldk, Vt, ldvt, O, ldo, B, Lq, Lk,
                        n_heads, static_cast<float*>(split_ws), split_ws_bytes, stream);
  GUARD_END
}

dif_status dif_attention_ex_static(int32_t dtype, int32_t head_dim, int32_t flags, const void* Q,
                                   int64_t ldq, const void* K, int64_t ldk, const void* Vt,
                                   int64_t ldvt, void* O, int64_t ldo, int32_t B, int32_t Lq,
                                   int32_t Lk, int32_t n_heads, dif_stream stream) {
  GUARD_BEGIN
  float* part = nullptr;
  size_t bytes = 0;
  const hipError_t e = dif::attention_static_scratch(&part, &bytes);
  if (e != hipSuccess)
    return fail(DIF_E_HIP, "static split workspace: %s", hipGetErrorString(e));
  if (head_dim == 64 || head_dim == 128) {
    if (dif::attention_split_bytes(head_dim) > bytes)
      return fail(DIF_E_WORKSPACE, "static split workspace %zu bytes < required %zu", bytes,
                  dif::attention_split_bytes(head_dim));
  }
  return attention_call(dtype, head_dim, flags, Q, ldq, K, ldk, Vt, ldvt, O, ldo, B, Lq, Lk,
                        n_heads, part, bytes, stream);
  GUARD_END
}

dif_status dif_mfma_probe(int32_t shape, int32_t iters, float* sink, double* flops,
                          dif_stream stream) {
  GUARD_BEGIN
  if (shape < 0 || shape > 2) return fail(DIF_E_ARG, "shape %d is not 0, 1 or 2", shape);
  if (iters < 1 || iters > 10000000) return fail(DIF_E_ARG, "iters %d outside 1 .. 10^7", iters);
  if (!sink || !flops) return fail(DIF_E_ARG, "null argument");
  if (!is_gfx950()) return fail(DIF_E_UNSUPPORTED, "current HIP device is not gfx950");
  int dev = 0, ncu = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
  HIP_TRY(dif::launch_mfma_probe(shape, iters, sink, ncu, static_cast<hipStream_t>(stream), flops));
  return DIF_OK;
  GUARD_END
}

dif_status dif_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = on != 0;
  return DIF_OK;
}

dif_status dif_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.recs.clear();
  g_prof.used = 0;
  return DIF_OK;
}

const char* dif_profile_kind_name(int32_t kind) {
  return (kind >= 0 && kind < DIF_PROF_KINDS) ? kKindNames[kind] : "";
}

dif_status dif_profile_collect(int64_t* launches, double* total_ms, double* flops, double* bytes) {
  GUARD_BEGIN
  if (!launches || !total_ms || !flops || !bytes) return fail(DIF_E_ARG, "null argument");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  for (int k = 0; k < DIF_PROF_KINDS; ++k) {
    launches[k] = 0;
    total_ms[k] = flops[k] = bytes[k] = 0.0;
  }
  for (const ProfRec& r : g_prof.recs) {
    HIP_TRY(hipEventSynchronize(r.b));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
    launches[r.kind] += 1;
    total_ms[r.kind] += ms;
    flops[r.kind] += r.flops;
    bytes[r.kind] += r.bytes;
  }
  return DIF_OK;
  GUARD_END
}

}  // extern "C"
