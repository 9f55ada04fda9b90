// Drives libdif's C ABI on the CPU (HIP runtime and kernel launches replaced
// by hip_host_stub.cpp, device memory = host memory) under AddressSanitizer
// and UndefinedBehaviorSanitizer: validation, plan layout of both plan kinds,
// workspace and text-cache carving, the timestep bound to a plan, and the
// error codes of every entry point.  Prints one line per case and exits
// non-zero on the first failed expectation.  Test infrastructure only.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "../../include/dif.h"

extern "C" long g_stub_launches;

namespace {

int g_fail = 0;

#define EXPECT(cond)                                                                \
  do {                                                                              \
    if (!(cond)) {                                                                  \
      std::fprintf(stderr, "FAIL %s:%d: %s (last error: %s)\n", __FILE__, __LINE__, \
                   #cond, dif_last_error());                                        \
      std::exit(1);                                                                 \
    }                                                                               \
  } while (0)

// 256-byte aligned host blocks ("device" memory), freed at exit
struct Arena {
  std::vector<void*> blocks;
  void* get(size_t bytes) {
    void* p = std::aligned_alloc(256, (bytes + 255) / 256 * 256);
    EXPECT(p != nullptr);
    std::memset(p, 0, (bytes + 255) / 256 * 256);
    blocks.push_back(p);
    return p;
  }
  ~Arena() {
    for (void* p : blocks) std::free(p);
  }
};

struct Model {
  dif_config cfg{};
  std::vector<dif_layer_weights> layers;
  dif_weights w{};
  dif_model* m = nullptr;
};

Model make_model(Arena& ar, int dtype, int D, int H, int dh, int F, int N, int gf, int gh, int gw,
                 int Lc) {
  Model M;
  dif_config& c = M.cfg;
  c.dim = D;
  c.n_heads = H;
  c.head_dim = dh;
  c.ffn_dim = F;
  c.n_layers = N;
  c.patch_dim = 64;
  c.freq_dim = 256;
  c.grid_f = gf;
  c.grid_h = gh;
  c.grid_w = gw;
  c.max_text_len = Lc;
  c.dtype = dtype;
  c.eps = 1e-6f;
  c.rope_theta = 1e4f;
  const size_t es = dtype == DIF_BF16 ? 2 : 4;
  auto mat = [&](size_t r, size_t k) { return ar.get(r * k * es); };
  auto vec = [&](size_t n) { return static_cast<const float*>(ar.get(n * 4)); };
  M.layers.resize(N);
  for (auto& L : M.layers) {
    L.mod = vec(6 * D);
    L.self_wq = mat(D, D);
    L.self_wk = mat(D, D);
    L.self_wv = mat(D, D);
    L.self_wo = mat(D, D);
    L.self_bq = vec(D);
    L.self_bk = vec(D);
    L.self_bv = vec(D);
    L.self_bo = vec(D);
    L.self_gq = vec(D);
    L.self_gk = vec(D);
    L.norm3_w = vec(D);
    L.norm3_b = vec(D);
    L.cross_wq = mat(D, D);
    L.cross_wk = mat(D, D);
    L.cross_wv = mat(D, D);
    L.cross_wo = mat(D, D);
    L.cross_bq = vec(D);
    L.cross_bk = vec(D);
    L.cross_bv = vec(D);
    L.cross_bo = vec(D);
    L.cross_gq = vec(D);
    L.cross_gk = vec(D);
    L.ffn_w1 = mat(F, D);
    L.ffn_b1 = vec(F);
    L.ffn_w2 = mat(D, F);
    L.ffn_b2 = vec(D);
  }
  M.w.patch_w = mat(D, 64);
  M.w.patch_b = vec(D);
  M.w.t_w1 = mat(D, 256);
  M.w.t_b1 = vec(D);
  M.w.t_w2 = mat(D, D);
  M.w.t_b2 = vec(D);
  M.w.t_w3 = mat(6 * D, D);
  M.w.t_b3 = vec(6 * D);
  M.w.head_mod = vec(2 * D);
  M.w.head_w = mat(64, D);
  M.w.head_b = vec(64);
  M.w.layers = M.layers.data();
  EXPECT(dif_model_create(&M.cfg, &M.w, &M.m) == DIF_OK);
  return M;
}

struct Masks {
  std::vector<uint8_t> block, self, cross, ffn;
  dif_step_masks s{};
};

// Seeded masks: per layer a random count of kept heads (0..H) and channels
// (0..F, whole 8-channel chunks on odd layers, single channels on even ones);
// layer 1 is gated off when n_layers > 2.
Masks make_masks(const dif_config& c, unsigned seed) {
  std::mt19937 g(seed);
  Masks m;
  const int N = c.n_layers, H = c.n_heads, F = c.ffn_dim;
  m.block.assign(N, 1);
  if (N > 2) m.block[1] = 0;
  m.self.assign((size_t)N * H, 0);
  m.cross.assign((size_t)N * H, 0);
  m.ffn.assign((size_t)N * F, 0);
  for (int l = 0; l < N; ++l) {
    for (int h = 0; h < H; ++h) {
      m.self[(size_t)l * H + h] = (g() % 4) != 0;
      m.cross[(size_t)l * H + h] = (g() % 3) != 0;
    }
    if (l % 2) {
      for (int ch = 0; ch < F / 8; ++ch) {
        const uint8_t k = (g() % 5) != 0;
        for (int e = 0; e < 8; ++e) m.ffn[(size_t)l * F + ch * 8 + e] = k;
      }
    } else {
      for (int j = 0; j < F; ++j) m.ffn[(size_t)l * F + j] = (g() % 3) != 0;
    }
  }
  // edge layers: everything pruned in layer 0 of odd seeds
  if (seed % 2) {
    std::fill(m.self.begin(), m.self.begin() + H, 0);
    std::fill(m.cross.begin(), m.cross.begin() + H, 0);
    std::fill(m.ffn.begin(), m.ffn.begin() + F, 0);
  }
  m.s = {m.block.data(), m.self.data(), m.cross.data(), m.ffn.data()};
  return m;
}

void validation_cases() {
  dif_config c{256, 4, 64, 1024, 2, 64, 256, 2, 8, 8, 16, DIF_F32, 1e-6f, 1e4f};
  EXPECT(dif_validate_config(&c) == DIF_OK);
  EXPECT(dif_validate_config(nullptr) == DIF_E_ARG);
  dif_config b = c;
  b.dim = 250;
  EXPECT(dif_validate_config(&b) == DIF_E_SHAPE);
  b = c;
  b.head_dim = 96;
  b.dim = 384;
  EXPECT(dif_validate_config(&b) == DIF_E_UNSUPPORTED);
  b = c;
  b.dtype = 7;
  EXPECT(dif_validate_config(&b) == DIF_E_ARG);
  b = c;
  b.grid_w = 0;
  EXPECT(dif_validate_config(&b) == DIF_E_SHAPE);
  b = c;
  b.eps = 0.f;
  EXPECT(dif_validate_config(&b) == DIF_E_ARG);
  Masks m = make_masks(c, 2);
  EXPECT(dif_validate_masks(&c, &m.s) == DIF_OK);
  m.ffn[5] = 2;
  EXPECT(dif_validate_masks(&c, &m.s) == DIF_E_MASK);
  EXPECT(std::strstr(dif_last_error(), "ffn_keep[5]") != nullptr);
  dif_step_masks nul{};
  EXPECT(dif_validate_masks(&c, &nul) == DIF_E_MASK);
  std::printf("ok validation\n");
}

void plan_cases(Arena& ar, int dtype, int D, int H, int dh, int F, int N, int gf, int gh, int gw,
                int Lc) {
  Model M = make_model(ar, dtype, D, H, dh, F, N, gf, gh, gw, Lc);
  const dif_config& c = M.cfg;
  const int L = gf * gh * gw;
  const char* dt = dtype == DIF_BF16 ? "bf16" : "f32";
  for (unsigned seed = 1; seed <= 4; ++seed) {
    Masks mk = make_masks(c, seed);
    for (int kind = 0; kind < 2; ++kind) {
      size_t bytes = 0;
      EXPECT(dif_plan_bytes_ex(M.m, &mk.s, kind, &bytes) == DIF_OK);
      void* mem = ar.get(bytes);
      dif_plan* p = nullptr;
      // too small / misaligned plan memory
      EXPECT(dif_plan_step_ex(M.m, 0, 999.f, &mk.s, kind, 0, mem, bytes - 1, nullptr, &p) ==
             DIF_E_WORKSPACE);
      EXPECT(dif_plan_step_ex(M.m, 0, 999.f, &mk.s, kind, 0, (char*)mem + 16, bytes, nullptr, &p) ==
             DIF_E_WORKSPACE);
      EXPECT(dif_plan_step_ex(M.m, 0, NAN, &mk.s, kind, 0, mem, bytes, nullptr, &p) == DIF_E_ARG);
      EXPECT(dif_plan_step_ex(M.m, 0, 999.f, &mk.s, kind, 4, mem, bytes, nullptr, &p) == DIF_E_ARG);
      EXPECT(dif_plan_step_ex(M.m, 0, 999.f, &mk.s, 5, 0, mem, bytes, nullptr, &p) == DIF_E_ARG);
      EXPECT(dif_plan_step_ex(M.m, 4096, 999.f, &mk.s, kind, 0, mem, bytes, nullptr, &p) == DIF_E_ARG);
      const float ts = 750.f;
      EXPECT(dif_plan_step_ex(M.m, 1, ts, &mk.s, kind, 0, mem, bytes, nullptr, &p) == DIF_OK);
      float t_got = 0.f;
      int32_t fl = -1;
      EXPECT(dif_plan_timestep(p, &t_got, &fl) == DIF_OK && t_got == ts && fl == 0);
      for (int l = 0; l < N; ++l) {
        dif_layer_info info{};
        EXPECT(dif_plan_layer_info(p, l, &info) == DIF_OK);
        int h = 0, hc = 0, f = 0;
        for (int i = 0; i < H; ++i) {
          h += mk.self[(size_t)l * H + i];
          hc += mk.cross[(size_t)l * H + i];
        }
        for (int j = 0; j < F; ++j) f += mk.ffn[(size_t)l * F + j];
        EXPECT(info.block_keep == mk.block[l] && info.self_heads == h && info.cross_heads == hc &&
               info.ffn_channels == f && info.ffn_padded % 64 == 0 && info.ffn_padded >= f);
      }
      dif_layer_info info{};
      EXPECT(dif_plan_layer_info(p, N, &info) == DIF_E_ARG);

      size_t wsb = 0;
      const int B = 2;
      EXPECT(dif_workspace_bytes(M.m, B, L, Lc, &wsb) == DIF_OK);
      void* ws = ar.get(wsb);
      const int Cp = 64;
      float* z = static_cast<float*>(ar.get((size_t)B * L * Cp * 4));
      float* v = static_cast<float*>(ar.get((size_t)B * L * Cp * 4));
      void* ctx = ar.get((size_t)B * Lc * D * (dtype == DIF_BF16 ? 2 : 4));
      // the timestep must be the plan's
      const long before = g_stub_launches;
      EXPECT(dif_step_forward(p, z, 500.f, ctx, B, L, Lc, v, ws, wsb, nullptr) == DIF_E_ARG);
      EXPECT(std::strstr(dif_last_error(), "t_s") != nullptr);
      EXPECT(g_stub_launches == before);
      EXPECT(dif_step_forward(p, z, ts, ctx, B, L, Lc, v, ws, wsb, nullptr) == DIF_OK);
      EXPECT(g_stub_launches > before);
      // workspace, shape and pointer errors
      EXPECT(dif_step_forward(p, z, ts, ctx, B, L, Lc, v, ws, wsb - 1, nullptr) == DIF_E_WORKSPACE);
      EXPECT(dif_step_forward(p, z, ts, ctx, B, L + 1, Lc, v, ws, wsb, nullptr) == DIF_E_SHAPE);
      EXPECT(dif_step_forward(p, z, ts, ctx, B, L, Lc + 1, v, ws, wsb, nullptr) == DIF_E_SHAPE);
      EXPECT(dif_step_forward(p, nullptr, ts, ctx, B, L, Lc, v, ws, wsb, nullptr) == DIF_E_ARG);
      EXPECT(dif_step_forward(p, z, INFINITY, ctx, B, L, Lc, v, ws, wsb, nullptr) == DIF_E_ARG);
      // every block on its own, and the block argument errors
      void* x = ar.get((size_t)B * L * D * (dtype == DIF_BF16 ? 2 : 4));
      float* e0 = static_cast<float*>(ar.get(6 * (size_t)D * 4));
      for (int l = 0; l < N; ++l)
        EXPECT(dif_block_forward(p, l, x, ctx, e0, B, L, Lc, ws, wsb, nullptr) == DIF_OK);
      EXPECT(dif_block_forward(p, N, x, ctx, e0, B, L, Lc, ws, wsb, nullptr) == DIF_E_ARG);
      EXPECT(dif_block_forward(p, 0, x, ctx, e0, B, L, Lc, (char*)ws + 64, wsb - 64, nullptr) ==
             DIF_E_WORKSPACE);
      // text cache: build, cached calls, errors
      size_t cb = 0;
      EXPECT(dif_text_cache_bytes(M.m, B, Lc, &cb) == DIF_OK);
      void* cache = ar.get(cb);
      EXPECT(dif_text_cache_build(M.m, ctx, B, Lc, cache, cb, nullptr) == DIF_OK);
      EXPECT(dif_text_cache_build(M.m, ctx, B, Lc, cache, cb - 1, nullptr) == DIF_E_WORKSPACE);
      EXPECT(dif_text_cache_bytes(M.m, B, Lc + 1, &cb) == DIF_E_SHAPE);
      EXPECT(dif_text_cache_bytes(M.m, B, Lc, &cb) == DIF_OK);
      for (int l = 0; l < N; ++l)
        EXPECT(dif_block_forward_cached(p, l, x, cache, cb, e0, B, L, Lc, ws, wsb, nullptr) == DIF_OK);
      EXPECT(dif_step_forward_cached(p, z, ts, cache, cb, B, L, Lc, v, ws, wsb, nullptr) == DIF_OK);
      EXPECT(dif_step_forward_cached(p, z, 1.f, cache, cb, B, L, Lc, v, ws, wsb, nullptr) == DIF_E_ARG);
      // rollouts check every timestep against its plan before launching
      const dif_plan* plans[2] = {p, p};
      const float good[2] = {ts, ts}, bad[2] = {ts, 250.f};
      float* eps0 = static_cast<float*>(ar.get((size_t)B * L * Cp * 4));
      const float* eps[2] = {eps0, eps0};
      const long b2 = g_stub_launches;
      EXPECT(dif_rollout(plans, bad, 2, DIF_SAMPLER_EULER, z, nullptr, ctx, B, L, Lc, v, ws, wsb,
                         nullptr) == DIF_E_ARG);
      EXPECT(dif_rollout_cached(plans, bad, 2, DIF_SAMPLER_RENOISE, z, eps, cache, cb, B, L, Lc, v,
                                ws, wsb, nullptr) == DIF_E_ARG);
      EXPECT(g_stub_launches == b2);
      EXPECT(dif_rollout(plans, good, 2, DIF_SAMPLER_RENOISE, z, eps, ctx, B, L, Lc, v, ws, wsb,
                         nullptr) == DIF_OK);
      EXPECT(dif_rollout(plans, good, 2, DIF_SAMPLER_RENOISE, z, nullptr, ctx, B, L, Lc, v, ws, wsb,
                         nullptr) == DIF_E_ARG);
      EXPECT(dif_rollout(plans, good, 2, 9, z, nullptr, ctx, B, L, Lc, v, ws, wsb, nullptr) ==
             DIF_E_ARG);
      EXPECT(dif_plan_destroy(p) == DIF_OK);

      // a plan built with DIF_PLAN_ANY_T accepts any timestep
      EXPECT(dif_plan_step_ex(M.m, 2, NAN, &mk.s, kind, DIF_PLAN_ANY_T, mem, bytes, nullptr, &p) ==
             DIF_OK);
      EXPECT(dif_plan_timestep(p, &t_got, &fl) == DIF_OK && fl == DIF_PLAN_ANY_T);
      EXPECT(dif_step_forward(p, z, 123.f, ctx, B, L, Lc, v, ws, wsb, nullptr) == DIF_OK);
      const dif_plan* any[2] = {p, p};
      EXPECT(dif_rollout(any, bad, 2, DIF_SAMPLER_EULER, z, nullptr, ctx, B, L, Lc, v, ws, wsb,
                         nullptr) == DIF_OK);
      EXPECT(dif_plan_destroy(p) == DIF_OK);
    }
  }
  // time embedding needs a workspace
  size_t wsb = 0;
  EXPECT(dif_workspace_bytes(M.m, 1, 1, 1, &wsb) == DIF_OK);
  void* ws = ar.get(wsb);
  float* e = static_cast<float*>(ar.get((size_t)D * 4));
  float* e0 = static_cast<float*>(ar.get(6 * (size_t)D * 4));
  EXPECT(dif_time_embed(M.m, 999.f, e, e0, ws, wsb, nullptr) == DIF_OK);
  EXPECT(dif_time_embed(M.m, 999.f, e, e0, ws, 0, nullptr) == DIF_E_WORKSPACE);
  // FFN reorder: the stub norms put channel j at (7 j) mod F, so the
  // permutation sorts by that key, descending
  std::vector<int32_t> perm(F);
  void* w1 = ar.get((size_t)F * D * (dtype == DIF_BF16 ? 2 : 4));
  void* w2 = ar.get((size_t)F * D * (dtype == DIF_BF16 ? 2 : 4));
  float* b1 = static_cast<float*>(ar.get((size_t)F * 4));
  void* scratch = ar.get((size_t)F * 12);
  EXPECT(dif_ffn_reorder(M.m, 0, w1, b1, w2, perm.data(), scratch, (size_t)F * 12, nullptr) == DIF_OK);
  for (int i = 1; i < F; ++i) EXPECT((perm[i - 1] * 7) % F >= (perm[i] * 7) % F);
  EXPECT(dif_ffn_reorder(M.m, 0, w1, b1, w2, perm.data(), scratch, (size_t)F * 12 - 1, nullptr) ==
         DIF_E_WORKSPACE);
  EXPECT(dif_ffn_reorder(M.m, N, w1, b1, w2, perm.data(), scratch, (size_t)F * 12, nullptr) == DIF_E_ARG);
  EXPECT(dif_model_destroy(M.m) == DIF_OK);
  std::printf("ok plans %s D=%d H=%d F=%d N=%d L=%d Lc=%d\n", dt, D, H, F, N, L, Lc);
}

void operator_cases(Arena& ar) {
  // dif_gemm argument errors
  void* A = ar.get(256 * 128 * 2);
  void* Bm = ar.get(256 * 128 * 2);
  void* Cm = ar.get(256 * 256 * 4);
  EXPECT(dif_gemm(DIF_BF16, DIF_BF16, A, 128, Bm, 128, Cm, 256, 256, 256, 128, DIF_EPI_STORE,
                  nullptr, nullptr, nullptr, nullptr) == DIF_OK);
  EXPECT(dif_gemm(DIF_BF16, DIF_BF16, A, 128, Bm, 128, Cm, 256, 256, 256, 100, 0, nullptr, nullptr,
                  nullptr, nullptr) == DIF_E_SHAPE);
  EXPECT(dif_gemm(DIF_BF16, DIF_BF16, A, 128, Bm, 128, Cm, 100, 256, 256, 128, 0, nullptr, nullptr,
                  nullptr, nullptr) == DIF_E_SHAPE);
  EXPECT(dif_gemm(DIF_BF16, 9, A, 128, Bm, 128, Cm, 256, 256, 256, 128, 0, nullptr, nullptr,
                  nullptr, nullptr) == DIF_E_ARG);
  EXPECT(dif_gemm(DIF_BF16, DIF_BF16, A, 128, Bm, 128, Cm, 256, 256, 256, 128, 3, nullptr, nullptr,
                  nullptr, nullptr) == DIF_E_ARG);
  EXPECT(dif_gemm(DIF_BF16, DIF_BF16, (char*)A + 2, 128, Bm, 128, Cm, 256, 256, 256, 128, 0, nullptr,
                  nullptr, nullptr, nullptr) == DIF_E_ARG);
  // the MFMA-rate probe: FLOP count, argument errors
  {
    float* sink = static_cast<float*>(ar.get(sizeof(float)));
    double fl = 0;
    EXPECT(dif_mfma_probe(0, 5, sink, &fl, nullptr) == DIF_OK && fl > 0);
    EXPECT(dif_mfma_probe(1, 5, sink, &fl, nullptr) == DIF_OK && fl > 0);
    EXPECT(dif_mfma_probe(2, 5, sink, &fl, nullptr) == DIF_OK && fl > 0);
    EXPECT(dif_mfma_probe(3, 5, sink, &fl, nullptr) == DIF_E_ARG);
    EXPECT(dif_mfma_probe(-1, 5, sink, &fl, nullptr) == DIF_E_ARG);
    EXPECT(dif_mfma_probe(0, 0, sink, &fl, nullptr) == DIF_E_ARG);
    EXPECT(dif_mfma_probe(0, 10000001, sink, &fl, nullptr) == DIF_E_ARG);
    EXPECT(dif_mfma_probe(0, 5, nullptr, &fl, nullptr) == DIF_E_ARG);
    EXPECT(dif_mfma_probe(0, 5, sink, nullptr, nullptr) == DIF_E_ARG);
  }
  // attention: plain and the block's launch (pre-scaled queries, split workspace)
  const int Bn = 1, L = 300, H = 3, dh = 128;
  void* Q = ar.get((size_t)L * H * dh * 2);
  void* K = ar.get((size_t)L * H * dh * 2);
  void* Vt = ar.get((size_t)H * dh * 320 * 2);
  void* O = ar.get((size_t)L * H * dh * 2);
  EXPECT(dif_attention(DIF_BF16, dh, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L, H, nullptr) ==
         DIF_OK);
  size_t sb = 0;
  EXPECT(dif_attention_split_bytes(dh, &sb) == DIF_OK && sb > 0);
  EXPECT(dif_attention_split_bytes(96, &sb) == DIF_E_UNSUPPORTED);
  EXPECT(dif_attention_split_bytes(dh, &sb) == DIF_OK);
  void* part = ar.get(sb);
  EXPECT(dif_attention_ex(DIF_BF16, dh, DIF_ATTN_Q_PRESCALED, Q, H * dh, K, H * dh, Vt, 320, O,
                          H * dh, Bn, L, L, H, part, sb, nullptr) == DIF_OK);
  EXPECT(dif_attention_ex(DIF_BF16, dh, 2, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L, H,
                          part, sb, nullptr) == DIF_E_ARG);
  EXPECT(dif_attention_ex(DIF_BF16, dh, 0, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L, H,
                          part, sb - 1, nullptr) == DIF_E_WORKSPACE);
  EXPECT(dif_attention_ex(DIF_BF16, dh, 0, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L, H,
                          (char*)part + 128, sb, nullptr) == DIF_E_WORKSPACE);
  EXPECT(dif_attention_ex_static(DIF_BF16, dh, DIF_ATTN_Q_PRESCALED, Q, H * dh, K, H * dh, Vt, 320,
                                 O, H * dh, Bn, L, L, H, nullptr) == DIF_OK);
  EXPECT(dif_attention_ex_static(DIF_BF16, 96, 0, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L,
                                 H, nullptr) == DIF_E_UNSUPPORTED);
  EXPECT(dif_attention(DIF_BF16, dh, Q, H * dh, K, H * dh, Vt, 200, O, H * dh, Bn, L, L, H, nullptr) ==
         DIF_E_SHAPE);
  EXPECT(dif_attention(DIF_BF16, dh, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, 0, H, nullptr) ==
         DIF_E_SHAPE);
  // hard gates: strict comparisons
  dif_config c{256, 2, 128, 64, 2, 64, 256, 1, 2, 2, 8, DIF_BF16, 1e-6f, 1e4f};
  std::vector<float> mb = {0.5f, 0.f}, ms(2 * 256, 0.f), mc(2 * 256, 0.f), mf(2 * 8, 0.f);
  ms[0] = 1.f;            // layer 0 head 0: mean > 0
  ms[128] = -1.f;         // layer 0 head 1: mean < 0
  mc[256 + 130] = NAN;    // layer 1 cross head 1: NaN prunes
  mf[3] = 1e-30f;         // layer 0 chunk 3
  std::vector<uint8_t> bk(2), sk(4), ck(4), fk(2 * 64);
  EXPECT(dif_hard_gates(&c, 8, mb.data(), ms.data(), mc.data(), mf.data(), bk.data(), sk.data(),
                        ck.data(), fk.data()) == DIF_OK);
  EXPECT(bk[0] == 1 && bk[1] == 0 && sk[0] == 1 && sk[1] == 0 && ck[3] == 0);
  for (int j = 0; j < 64; ++j) EXPECT(fk[j] == (j / 8 == 3 ? 1 : 0));
  EXPECT(dif_hard_gates(&c, 7, mb.data(), ms.data(), mc.data(), mf.data(), bk.data(), sk.data(),
                        ck.data(), fk.data()) == DIF_E_SHAPE);
  // kernel timing over the stub events
  EXPECT(dif_profile_reset() == DIF_OK && dif_profile_enable(1) == DIF_OK);
  EXPECT(dif_attention(DIF_BF16, dh, Q, H * dh, K, H * dh, Vt, 320, O, H * dh, Bn, L, L, H, nullptr) ==
         DIF_OK);
  EXPECT(dif_profile_enable(0) == DIF_OK);
  int64_t la[DIF_PROF_KINDS];
  double ms_[DIF_PROF_KINDS], fl[DIF_PROF_KINDS], by[DIF_PROF_KINDS];
  EXPECT(dif_profile_collect(la, ms_, fl, by) == DIF_OK);
  EXPECT(la[1] == 1 && std::string(dif_profile_kind_name(1)) == "attn_self");
  EXPECT(std::fabs(fl[1] - 4.0 * L * L * dh * H) < 1.0);
  std::printf("ok operators\n");
}

}  // namespace

int main() {
  Arena ar;
  validation_cases();
  // float32, head 64 (the tiny stack's shapes) and bfloat16, head 128 with a
  // ragged token count and several text lengths
  plan_cases(ar, DIF_F32, 256, 4, 64, 1024, 3, 2, 8, 8, 16);
  plan_cases(ar, DIF_BF16, 512, 4, 128, 1000, 3, 3, 5, 7, 77);
  plan_cases(ar, DIF_F32, 256, 2, 128, 96, 2, 1, 3, 5, 5);
  operator_cases(ar);
  std::printf("harness: all cases passed\n");
  return g_fail;
}
