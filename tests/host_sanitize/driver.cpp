// Runs every entry point of the C ABI on the CPU against the host stand-ins of the kernel
// launchers (stub_kernels.cpp), under AddressSanitizer and UndefinedBehaviorSanitizer: valid
// calls over bf16 and fp32 storage, sliding windows, block-causal masks, precise attention I/O,
// KV-head subsets, packed W_dS, batches past the fused work-list limit and empty contexts, each
// with a workspace of exactly the queried size; then rejected calls (short or misaligned
// workspace, NULL pointers, bad sizes), which must return their error code and enqueue
// nothing; then the workspace queries at serving sizes and at the limits of every size; then
// 300 seeded random configurations (a sixth of them outside the documented shapes), each call
// accepted with every extent in bounds or refused with nothing enqueued.
// Prints one line per case; exits non-zero on the first failed expectation.
#include <climits>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "hspec.h"
#include "stub_registry.h"

namespace {

int g_cases = 0;

[[noreturn]] void fail_case(const char* what, int got, int want) {
  std::fprintf(stderr, "FAIL %s: status %d, expected %d (%s)\n", what, got, want, hspec_last_error());
  std::exit(1);
}

void expect(const char* what, hspec_status got, hspec_status want) {
  ++g_cases;
  if (got != want) fail_case(what, (int)got, (int)want);
  if (want != HSPEC_OK && hspec_last_error()[0] == 0) {
    std::fprintf(stderr, "FAIL %s: error without a message\n", what);
    std::exit(1);
  }
  if (want == HSPEC_OK && hspec_last_error()[0] != 0) {
    std::fprintf(stderr, "FAIL %s: success left the message '%s'\n", what, hspec_last_error());
    std::exit(1);
  }
  std::printf("ok   %-60s -> %d\n", what, (int)got);
}

// A rejected call must enqueue nothing.
template <class F>
void expect_reject(const char* what, hspec_status want, F&& call) {
  const long before = stub_launches();
  expect(what, call(), want);
  if (stub_launches() != before) {
    std::fprintf(stderr, "FAIL %s: a rejected call launched %ld kernels\n", what, stub_launches() - before);
    std::exit(1);
  }
}

// "Device" memory: host memory of exactly `bytes`, 256-byte aligned, registered with the stubs.
struct Pool {
  std::vector<void*> bufs;
  void* get(size_t bytes) {
    void* p = nullptr;
    if (posix_memalign(&p, 256, bytes ? bytes : 1)) std::abort();
    std::memset(p, 0, bytes ? bytes : 1);
    stub_register(p, bytes);
    bufs.push_back(p);
    return p;
  }
  ~Pool() {
    for (void* p : bufs) {
      stub_unregister(p);
      std::free(p);
    }
  }
};

size_t esz(hspec_dtype d) { return d == HSPEC_F32 ? 4 : 2; }

struct MambaW {
  hspec_mamba_w w{};
};
MambaW make_mamba(Pool& pool, const hspec_mamba_cfg& c) {
  const size_t s = esz(c.dtype), di = (size_t)c.H * c.P, gn = (size_t)c.G * c.N, dS = di * c.N;
  const size_t dproj = 2 * di + 2 * gn + c.H, conv_dim = di + 2 * gn;
  MambaW m;
  m.w.W_r = pool.get((size_t)c.r * c.d_h * s);
  m.w.W_dS = pool.get(dS * c.r * s);
  m.w.W_in = pool.get(dproj * c.d_model * s);
  m.w.conv_w = pool.get(conv_dim * c.conv_w * s);
  m.w.conv_b = pool.get(conv_dim * s);
  m.w.dt_bias = (const float*)pool.get((size_t)c.H * 4);
  m.w.A_log = (const float*)pool.get((size_t)c.H * 4);
  m.w.D = (const float*)pool.get((size_t)c.H * 4);
  m.w.gnorm_w = (const float*)pool.get(di * 4);
  m.w.W_out = pool.get((size_t)c.d_model * di * s);
  return m;
}

hspec_attn_w make_attn(Pool& pool, const hspec_attn_cfg& c) {
  const size_t s = esz(c.dtype);
  hspec_attn_w w{};
  w.W_q = pool.get((size_t)c.Hq * c.D * c.d_model * s);
  w.W_k = pool.get((size_t)c.Hkv * c.D * c.d_model * s);
  w.W_v = pool.get((size_t)c.Hkv * c.D * c.d_model * s);
  w.W_o = pool.get((size_t)c.d_model * c.Hq * c.D * s);
  w.q_norm_w = (const float*)pool.get((size_t)c.D * 4);
  w.k_norm_w = (const float*)pool.get((size_t)c.D * 4);
  return w;
}

struct Paged {
  void *kc, *vc;
  int32_t *pt, *lens;
};
Paged make_paged(Pool& pool, const hspec_attn_cfg& c) {
  const int heads = c.Hkv_cache > 0 ? c.Hkv_cache : c.Hkv;
  const size_t cache = (size_t)c.num_pages * c.page_size * heads * c.D * esz(c.dtype);
  Paged p;
  p.kc = pool.get(cache);
  p.vc = pool.get(cache);
  p.pt = (int32_t*)pool.get((size_t)c.B * c.max_pages * 4);
  p.lens = (int32_t*)pool.get((size_t)c.B * 4);
  return p;
}

// The workspace of a call: exactly `bytes`.
void* workspace(Pool& pool, size_t bytes) {
  if (bytes == 0 || bytes % 256) {
    std::fprintf(stderr, "FAIL workspace query returned %zu\n", bytes);
    std::exit(1);
  }
  return pool.get(bytes);
}

hspec_attn_cfg attn_cfg(hspec_dtype dt, int B, int k, int d_model, int Hq, int Hkv, int D) {
  hspec_attn_cfg c{};
  c.B = B; c.k = k; c.d_model = d_model; c.Hq = Hq; c.Hkv = Hkv; c.D = D;
  c.page_size = 16; c.max_pages = 8; c.num_pages = 32; c.window = 0; c.split_tokens = 0;
  c.flags = 0; c.dtype = dt; c.eps = 1e-6f; c.scale = 0.f; c.rope_theta = 10000.0;
  c.Hkv_cache = 0; c.kv_heads = nullptr;
  return c;
}

hspec_mamba_cfg mamba_cfg(hspec_dtype dt, int B, int k, int d_model, int N) {
  hspec_mamba_cfg c{};
  c.B = B; c.k = k; c.d_model = d_model; c.d_h = 512; c.r = 64; c.H = 4; c.P = 64; c.N = N; c.G = 2;
  c.chunk = 4; c.conv_w = 4; c.flags = 0; c.dtype = dt; c.eps = 1e-6f;
  return c;
}

// ------------------------------------------------------------------------ valid calls

void run_attention_calls(const char* name, const hspec_attn_cfg& c, int max_ctx) {
  char what[160];
  Pool pool;
  const hspec_attn_w w = make_attn(pool, c);
  const Paged pg = make_paged(pool, c);
  const size_t s = esz(c.dtype), M = (size_t)c.B * c.k;
  void* x = pool.get(M * c.d_model * s);
  float* out = (float*)pool.get(M * c.d_model * 4);
  {
    const size_t n = hspec_target_kv_block_attn_workspace(&c, max_ctx);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: target_kv_block_attn", name);
    expect(what, hspec_target_kv_block_attn(&c, &w, x, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, ws, n, nullptr),
           HSPEC_OK);
    int32_t st = -1;
    std::snprintf(what, sizeof what, "%s: read_status", name);
    expect(what, hspec_read_status(ws, &st, nullptr), HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: target_kv_block_attn, workspace 256 bytes short", name);
    expect_reject(what, HSPEC_ERR_WORKSPACE, [&] {
      return hspec_target_kv_block_attn(&c, &w, x, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, ws, n - 256, nullptr);
    });
    std::snprintf(what, sizeof what, "%s: target_kv_block_attn, misaligned workspace", name);
    expect_reject(what, HSPEC_ERR_WORKSPACE, [&] {
      return hspec_target_kv_block_attn(&c, &w, x, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, (char*)ws + 64,
                                        n - 256, nullptr);
    });
    std::snprintf(what, sizeof what, "%s: target_kv_block_attn, NULL page table", name);
    expect_reject(what, HSPEC_ERR_NULL, [&] {
      return hspec_target_kv_block_attn(&c, &w, x, pg.kc, pg.vc, nullptr, pg.lens, max_ctx, out, ws, n, nullptr);
    });
  }
  {
    void* q = pool.get(M * c.Hq * c.D * s);
    void* kb = pool.get(M * c.Hkv * c.D * s);
    void* vb = pool.get(M * c.Hkv * c.D * s);
    float* o = (float*)pool.get(M * c.Hq * c.D * 4);
    const size_t n = hspec_paged_attn_workspace(&c, max_ctx);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: paged_attn", name);
    expect(what, hspec_paged_attn(&c, q, kb, vb, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, o, ws, n, nullptr), HSPEC_OK);
    const unsigned phases[] = {HSPEC_PHASE_WORKLIST, HSPEC_PHASE_SWEEP, HSPEC_PHASE_REDUCE,
                               HSPEC_PHASE_SWEEP | HSPEC_PHASE_REDUCE};
    for (unsigned ph : phases) {
      std::snprintf(what, sizeof what, "%s: paged_attn_phase %u", name, ph);
      expect(what, hspec_paged_attn_phase(&c, q, kb, vb, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, o, ws, n, ph, nullptr),
             HSPEC_OK);
    }
    std::snprintf(what, sizeof what, "%s: paged_attn_phase, unknown phase bit", name);
    expect_reject(what, HSPEC_ERR_UNSUPPORTED, [&] {
      return hspec_paged_attn_phase(&c, q, kb, vb, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, o, ws, n, 8u, nullptr);
    });
    if (max_ctx > 0) {
      int32_t* slots = (int32_t*)pool.get((size_t)c.B * max_ctx * 4);
      int32_t* st = (int32_t*)pool.get(4);
      std::snprintf(what, sizeof what, "%s: gather_slots", name);
      expect(what, hspec_gather_slots(c.B, c.max_pages, c.page_size, c.num_pages, pg.pt, pg.lens, max_ctx, slots, st,
                                      nullptr),
             HSPEC_OK);
    }
  }
}

void run_mamba_calls(const char* name, const hspec_mamba_cfg& c) {
  char what[160];
  Pool pool;
  MambaW m = make_mamba(pool, c);
  const size_t s = esz(c.dtype), M = (size_t)c.B * c.k, dS = (size_t)c.H * c.P * c.N;
  if (c.flags & HSPEC_W_DS_PACKED) {
    void* packed = pool.get(hspec_pack_w_ds_bytes((int)dS, c.r));
    std::snprintf(what, sizeof what, "%s: pack_w_ds", name);
    expect(what, hspec_pack_w_ds((int)dS, c.r, m.w.W_dS, packed, nullptr), HSPEC_OK);
    m.w.W_dS = packed;
  }
  void* h = pool.get((size_t)c.B * c.d_h * s);
  void* u = pool.get(M * c.d_model * s);
  float* out = (float*)pool.get(M * c.d_model * 4);
  float* S = (float*)pool.get((size_t)c.B * dS * 4);
  {
    const size_t n = hspec_state_init_workspace(&c);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: state_init", name);
    expect(what, hspec_state_init(&c, &m.w, h, S, ws, n, nullptr), HSPEC_OK);
  }
  {
    const size_t n = hspec_mamba_block_scan_workspace(&c);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: mamba_block_scan", name);
    expect(what, hspec_mamba_block_scan(&c, &m.w, h, u, out, S, ws, n, nullptr), HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: mamba_block_scan without S_final", name);
    expect(what, hspec_mamba_block_scan(&c, &m.w, h, u, out, nullptr, ws, n, nullptr), HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: mamba_block_scan, NULL W_in", name);
    hspec_mamba_w bad = m.w;
    bad.W_in = nullptr;
    expect_reject(what, HSPEC_ERR_NULL, [&] { return hspec_mamba_block_scan(&c, &bad, h, u, out, S, ws, n, nullptr); });
  }
  {
    const int T = c.k;
    void* x = pool.get(M * c.H * c.P * s);
    float* dt = (float*)pool.get(M * c.H * 4);
    float* A = (float*)pool.get((size_t)c.H * 4);
    void* Bm = pool.get(M * c.G * c.N * s);
    void* Cm = pool.get(M * c.G * c.N * s);
    float* Dk = (float*)pool.get((size_t)c.H * 4);
    void* S0 = pool.get((size_t)c.B * dS * s);
    float* y = (float*)pool.get(M * c.H * c.P * 4);
    const size_t n = hspec_ssd_scan_workspace(c.B, T, c.H, c.P, c.N, c.G, c.dtype);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: ssd_scan", name);
    expect(what, hspec_ssd_scan(c.B, T, c.H, c.P, c.N, c.G, c.chunk, c.dtype, x, dt, A, Bm, Cm, Dk, S0, y, S, ws, n,
                                nullptr),
           HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: ssd_scan from zeros", name);
    expect(what, hspec_ssd_scan(c.B, T, c.H, c.P, c.N, c.G, c.chunk, c.dtype, x, dt, A, Bm, Cm, Dk, nullptr, y,
                                nullptr, ws, n, nullptr),
           HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: ssd_scan, chunk 17", name);
    expect_reject(what, HSPEC_ERR_UNSUPPORTED, [&] {
      return hspec_ssd_scan(c.B, T, c.H, c.P, c.N, c.G, 17, c.dtype, x, dt, A, Bm, Cm, Dk, S0, y, S, ws, n, nullptr);
    });
  }
  {
    const int Ms[] = {1, 5, 64, 300};
    for (int Mm : Ms) {
      const int N = 96, K = 520;
      void* A = pool.get((size_t)Mm * K * s);
      void* W = pool.get((size_t)N * K * s);
      float* R = (float*)pool.get((size_t)Mm * N * 4);
      float* Cc = (float*)pool.get((size_t)Mm * N * 4);
      const size_t n = hspec_linear_workspace(c.dtype, Mm, N, K);
      void* ws = workspace(pool, n);
      std::snprintf(what, sizeof what, "%s: linear M=%d", name, Mm);
      expect(what, hspec_linear(c.dtype, Mm, N, K, A, W, R, Cc, ws, n, nullptr), HSPEC_OK);
      expect(what, hspec_linear(c.dtype, Mm, N, K, A, W, nullptr, Cc, ws, n, nullptr), HSPEC_OK);
    }
  }
}

void run_step_calls(const char* name, const hspec_mamba_cfg& mc, const hspec_attn_cfg& ac, int max_ctx) {
  char what[160];
  Pool pool;
  MambaW m = make_mamba(pool, mc);
  if (mc.flags & HSPEC_W_DS_PACKED) {
    const int dS = mc.H * mc.P * mc.N;
    void* packed = pool.get(hspec_pack_w_ds_bytes(dS, mc.r));
    expect("pack_w_ds", hspec_pack_w_ds(dS, mc.r, m.w.W_dS, packed, nullptr), HSPEC_OK);
    m.w.W_dS = packed;
  }
  const hspec_attn_w aw = make_attn(pool, ac);
  const Paged pg = make_paged(pool, ac);
  const size_t s = esz(mc.dtype), M = (size_t)mc.B * mc.k;
  const float* n1 = (const float*)pool.get((size_t)mc.d_model * 4);
  const float* n2 = (const float*)pool.get((size_t)mc.d_model * 4);
  const float* n3 = (const float*)pool.get((size_t)mc.d_model * 4);
  void* h = pool.get((size_t)mc.B * mc.d_h * s);
  void* e = pool.get(M * mc.d_model * s);
  float* out = (float*)pool.get(M * mc.d_model * 4);
  {
    const size_t n = hspec_draft_step_workspace(&mc, &ac, max_ctx);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: draft_step", name);
    expect(what, hspec_draft_step(&mc, &m.w, n1, &ac, &aw, n2, h, e, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, ws, n,
                                  nullptr),
           HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: draft_step, configs disagree on k", name);
    hspec_attn_cfg ac2 = ac;
    ac2.k = ac.k + 1;
    expect_reject(what, HSPEC_ERR_SHAPE, [&] {
      return hspec_draft_step(&mc, &m.w, n1, &ac2, &aw, n2, h, e, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, ws, n,
                              nullptr);
    });
  }
  {
    // three layers: Mamba + attention + MLP, attention + MLP, Mamba + MLP
    const int ff = 136;
    const void* Wg = pool.get((size_t)ff * mc.d_model * s);
    const void* Wu = pool.get((size_t)ff * mc.d_model * s);
    const void* Wd = pool.get((size_t)mc.d_model * ff * s);
    const Paged pg2 = make_paged(pool, ac);
    hspec_layer_w L[3] = {};
    for (auto& l : L) {
      l.norm1_w = n1; l.norm2_w = n2; l.norm3_w = n3; l.W_gate = Wg; l.W_up = Wu; l.W_down = Wd;
    }
    L[0].mamba = &m.w; L[0].attn = &aw; L[0].k_cache = pg.kc; L[0].v_cache = pg.vc;
    L[1].attn = &aw; L[1].k_cache = pg2.kc; L[1].v_cache = pg2.vc;
    L[2].mamba = &m.w;
    const size_t n = hspec_drafter_forward_workspace(&mc, &ac, ff, max_ctx);
    void* ws = workspace(pool, n);
    std::snprintf(what, sizeof what, "%s: drafter_forward (3 layers)", name);
    expect(what, hspec_drafter_forward(&mc, &ac, ff, 3, m.w.W_r, m.w.W_dS, L, h, e, pg.pt, pg.lens, max_ctx, out, ws,
                                       n, nullptr),
           HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: drafter_forward (one attention layer)", name);
    expect(what, hspec_drafter_forward(&mc, &ac, ff, 1, m.w.W_r, m.w.W_dS, L + 1, nullptr, e, pg.pt, pg.lens, max_ctx,
                                       out, ws, n, nullptr),
           HSPEC_OK);
    std::snprintf(what, sizeof what, "%s: drafter_forward, ff not a multiple of 8", name);
    expect_reject(what, HSPEC_ERR_UNSUPPORTED, [&] {
      return hspec_drafter_forward(&mc, &ac, ff + 4, 3, m.w.W_r, m.w.W_dS, L, h, e, pg.pt, pg.lens, max_ctx, out, ws,
                                   n, nullptr);
    });
  }
}

void run_inject_calls(const char* name, const hspec_attn_cfg& c) {
  char what[160];
  Pool pool;
  const int d_h = 384, nl = 2;
  const size_t s = esz(c.dtype), M = (size_t)c.B * c.k, kvw = (size_t)c.Hkv * c.D;
  void* h = pool.get(M * d_h * s);
  void* Wfc = pool.get((size_t)c.d_model * d_h * s);
  const void* Wk[nl];
  const void* Wv[nl];
  const float* kn[nl];
  void* kc[nl];
  void* vc[nl];
  Paged pg{};
  for (int l = 0; l < nl; ++l) {
    Wk[l] = pool.get(kvw * c.d_model * s);
    Wv[l] = pool.get(kvw * c.d_model * s);
    kn[l] = (const float*)pool.get((size_t)c.D * 4);
    pg = make_paged(pool, c);
    kc[l] = pg.kc;
    vc[l] = pg.vc;
  }
  const size_t n = hspec_kv_inject_workspace(&c, d_h);
  void* ws = workspace(pool, n);
  std::snprintf(what, sizeof what, "%s: kv_inject", name);
  expect(what, hspec_kv_inject(&c, d_h, nl, h, Wfc, Wk, Wv, kn, kc, vc, pg.pt, pg.lens, ws, n, nullptr), HSPEC_OK);
  hspec_attn_cfg sub = c;
  sub.Hkv_cache = c.Hkv + 1;
  std::snprintf(what, sizeof what, "%s: kv_inject with a KV-head subset", name);
  expect_reject(what, HSPEC_ERR_UNSUPPORTED, [&] {
    return hspec_kv_inject(&sub, d_h, nl, h, Wfc, Wk, Wv, kn, kc, vc, pg.pt, pg.lens, ws, n, nullptr);
  });
}

void run_head_calls() {
  Pool pool;
  hspec_head_cfg c{};
  c.B = 3; c.k = 5; c.d_model = 136; c.vocab = 1000; c.rank = 64; c.eps = 1e-6f; c.temperature = 0.7f;
  const size_t M = (size_t)c.B * c.k;
  hspec_head_w w{};
  w.norm_f_w = (const float*)pool.get((size_t)c.d_model * 4);
  w.W_lm = pool.get((size_t)c.vocab * c.d_model * 2);
  w.E_M = pool.get((size_t)c.vocab * c.rank * 2);
  w.U_M = pool.get((size_t)c.vocab * c.rank * 2);
  const float* hid = (const float*)pool.get(M * c.d_model * 4);
  const int32_t* prev = (const int32_t*)pool.get((size_t)c.B * 4);
  const float* gum = (const float*)pool.get(M * c.vocab * 4);
  const int32_t* forced = (const int32_t*)pool.get(M * 4);
  int32_t* tok = (int32_t*)pool.get(M * 4);
  float* logits = (float*)pool.get(M * c.vocab * 4);
  const size_t n = hspec_draft_head_workspace(&c);
  void* ws = workspace(pool, n);
  expect("draft_head greedy", hspec_draft_head(&c, &w, hid, prev, nullptr, nullptr, tok, nullptr, ws, n, nullptr),
         HSPEC_OK);
  expect("draft_head sampled, forced, logits",
         hspec_draft_head(&c, &w, hid, prev, gum, forced, tok, logits, ws, n, nullptr), HSPEC_OK);
  hspec_head_cfg cold = c;
  cold.temperature = 0.f;
  expect_reject("draft_head sampled at temperature 0", HSPEC_ERR_SHAPE, [&] {
    return hspec_draft_head(&cold, &w, hid, prev, gum, nullptr, tok, nullptr, ws, n, nullptr);
  });
  hspec_head_cfg odd = c;
  odd.rank = 48;
  expect_reject("draft_head rank 48", HSPEC_ERR_UNSUPPORTED, [&] {
    return hspec_draft_head(&odd, &w, hid, prev, nullptr, nullptr, tok, nullptr, ws, n, nullptr);
  });
}

// --------------------------------------------------------------- queries at the limits

void run_queries() {
  // serving sizes: 64 requests of up to 32768 cached positions, 8B-class target
  hspec_attn_cfg a = attn_cfg(HSPEC_BF16, 64, 16, 4096, 32, 8, 128);
  a.page_size = 16; a.max_pages = 2048; a.num_pages = 64 * 2048;
  hspec_mamba_cfg m = mamba_cfg(HSPEC_BF16, 64, 16, 4096, 128);
  m.d_h = 3 * 4096; m.r = 1024; m.H = 128; m.G = 8;
  const size_t step = hspec_draft_step_workspace(&m, &a, 32768);
  const size_t fwd = hspec_drafter_forward_workspace(&m, &a, 14336, 32768);
  std::printf("ok   serving-size queries: draft_step %zu bytes, drafter_forward %zu bytes\n", step, fwd);
  if (step == 0 || fwd < step) std::exit(1);
  // every query at the extremes of its sizes (a query never fails; it sizes what the call,
  // which validates first, would use)
  const int lens[] = {0, 1, 32767, 1 << 20, INT_MAX - 1, INT_MAX};
  for (int L : lens) {
    hspec_attn_cfg big = attn_cfg(HSPEC_F32, 32767, 128, 8, 128, 128, 128);
    big.window = L > 0 ? L : 0;
    (void)hspec_paged_attn_workspace(&big, L);
    (void)hspec_target_kv_block_attn_workspace(&big, L);
    big.window = 0;
    (void)hspec_paged_attn_workspace(&big, L);
    ++g_cases;
  }
  std::printf("ok   attention workspace queries at context lengths up to INT_MAX\n");
  (void)hspec_linear_workspace(HSPEC_F32, INT_MAX, INT_MAX, INT_MAX);
  (void)hspec_ssd_scan_workspace(INT_MAX, INT_MAX, INT_MAX, 64, 128, 1, HSPEC_F32);
  hspec_head_cfg h{};
  h.B = INT_MAX; h.k = INT_MAX; h.d_model = INT_MAX; h.vocab = INT_MAX; h.rank = 32;
  (void)hspec_draft_head_workspace(&h);
  (void)hspec_pack_w_ds_bytes(INT_MAX - 15, INT_MAX - 63);
  std::printf("ok   GEMM, scan, head and packing queries at INT_MAX sizes\n");
  // rejected configurations
  hspec_attn_cfg bad = attn_cfg(HSPEC_BF16, 2, 4, 64, 8, 2, 128);
  bad.split_tokens = 8192 + 64;
  expect_reject("paged_attn, split above the maximum", HSPEC_ERR_UNSUPPORTED, [&] {
    return hspec_paged_attn(&bad, (void*)1, (void*)1, (void*)1, (void*)1, (void*)1, (const int32_t*)1,
                            (const int32_t*)1, 100, (float*)1, (void*)256, 1 << 20, nullptr);
  });
  bad = attn_cfg(HSPEC_BF16, 2, 4, 64, 8, 2, 128);
  const int32_t heads[2] = {0, 5};
  bad.Hkv_cache = 4; bad.kv_heads = heads;
  expect_reject("paged_attn, KV head outside the cache", HSPEC_ERR_SHAPE, [&] {
    return hspec_paged_attn(&bad, (void*)1, (void*)1, (void*)1, (void*)1, (void*)1, (const int32_t*)1,
                            (const int32_t*)1, 100, (float*)1, (void*)256, 1 << 20, nullptr);
  });
  bad = attn_cfg(HSPEC_BF16, 2, 4, 64, 8, 2, 128);
  expect_reject("paged_attn, context of INT_MAX keys", HSPEC_ERR_UNSUPPORTED, [&] {
    return hspec_paged_attn(&bad, (void*)1, (void*)1, (void*)1, (void*)1, (void*)1, (const int32_t*)1,
                            (const int32_t*)1, INT_MAX, (float*)1, (void*)256, 1 << 20, nullptr);
  });
  for (int s = 0; s <= 7; ++s) ++g_cases, (void)hspec_status_string((hspec_status)s);   // 7: no such status
}

}  // namespace

// ------------------------------------------------------------ seeded random configurations

// Configurations drawn from a fixed seed over the shapes the ABI documents (and some it refuses).
// Every call is either accepted, with every extent a kernel would touch inside the caller's
// buffers and inside its workspace region (the stand-ins abort otherwise), or rejected with a
// message and nothing enqueued.
struct Lcg {
  unsigned long long s;
  int operator()(int n) {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return (int)((s >> 33) % (unsigned long long)n);
  }
  template <size_t K>
  int pick(const int (&v)[K]) { return v[(*this)((int)K)]; }
};

int g_rand_ok = 0, g_rand_rejected = 0;

void accepted_or_refused(const char* what, hspec_status got, long launches_before) {
  ++g_cases;
  if (got == HSPEC_OK) {
    if (hspec_last_error()[0] != 0) {
      std::fprintf(stderr, "FAIL %s: success left the message '%s'\n", what, hspec_last_error());
      std::exit(1);
    }
    ++g_rand_ok;
    return;
  }
  if (hspec_last_error()[0] == 0) {
    std::fprintf(stderr, "FAIL %s: error %d without a message\n", what, (int)got);
    std::exit(1);
  }
  if (stub_launches() != launches_before) {
    std::fprintf(stderr, "FAIL %s: a refused call launched %ld kernels\n", what, stub_launches() - launches_before);
    std::exit(1);
  }
  ++g_rand_rejected;
}

// Workspace of exactly the queried size, or (when the query gives none) a small one the call
// must refuse.
void* random_ws(Pool& pool, size_t n) { return pool.get(n > 0 ? n : 256); }

void run_random_calls(int count) {
  Lcg r{0x2609241970ull};
  static const int Bs[] = {1, 2, 3, 5, 8}, ks[] = {1, 3, 5, 8, 16}, dms[] = {64, 128, 256, 320};
  static const int Hs[] = {1, 2, 4, 5, 8, 12, 16}, Ns[] = {16, 32, 64, 128}, Ds[] = {64, 128};
  static const int Hkvs[] = {1, 2, 4, 8}, gs[] = {1, 2, 4, 8}, wins[] = {0, 0, 16, 64};
  static const int splits[] = {0, 0, 64, 128}, pages[] = {1, 2, 8, 20}, dhs[] = {128, 256}, rs[] = {64, 128};
  for (int i = 0; i < count; ++i) {
    char what[160];
    const hspec_dtype dt = r(6) ? HSPEC_BF16 : HSPEC_F32;
    const int B = r.pick(Bs), k = r.pick(ks), d_model = r.pick(dms);
    hspec_mamba_cfg mc = mamba_cfg(dt, B, k, d_model, r.pick(Ns));
    mc.H = r.pick(Hs);
    int G = 1 << r(3);
    while (mc.H % G) G >>= 1;
    mc.G = G;
    mc.chunk = 1 + r(16);
    mc.conv_w = r(4) ? 4 : 2 + r(5);
    mc.d_h = r.pick(dhs);
    mc.r = r.pick(rs);
    if (dt == HSPEC_BF16 && r(2)) mc.flags |= HSPEC_W_DS_PACKED;
    const int Hkv = r.pick(Hkvs), g = r.pick(gs);
    hspec_attn_cfg ac = attn_cfg(dt, B, k, d_model, Hkv * g, Hkv, r.pick(Ds));
    ac.window = r.pick(wins);
    ac.flags = (r(3) == 0 ? HSPEC_BLOCK_CAUSAL : 0u) | (r(4) == 0 ? HSPEC_ATTN_PRECISE_IO : 0u);
    ac.split_tokens = r.pick(splits);
    ac.max_pages = r.pick(pages);
    ac.num_pages = ac.max_pages * B + 3 * r(2);
    // about one draw in six leaves the documented shapes in one respect, which must be refused
    // before anything is enqueued
    switch (r(6) == 0 ? 1 + r(6) : 0) {
      case 1: mc.N = 48; break;
      case 2: ac.page_size = 8; break;
      case 3: ac.D = 96; break;
      case 4: ac.k = mc.k = 16; ac.Hq = ac.Hkv * 16; break;
      case 5: mc.chunk = 17; break;
      case 6: ac.d_model = mc.d_model = d_model + 4; break;
      default: break;
    }
    const int max_ctx = r(ac.max_pages * ac.page_size + 1);
    std::printf("     random %d: %s B=%d k=%d d=%d H=%d N=%d G=%d chunk=%d conv=%d packed=%d Hq=%d Hkv=%d D=%d "
                "win=%d flags=%u split=%d pages=%d max_ctx=%d\n",
                i, dt == HSPEC_BF16 ? "bf16" : "f32", B, mc.k, mc.d_model, mc.H, mc.N, mc.G, mc.chunk, mc.conv_w,
                (mc.flags & HSPEC_W_DS_PACKED) ? 1 : 0, ac.Hq, ac.Hkv, ac.D, ac.window, ac.flags, ac.split_tokens,
                ac.max_pages, max_ctx);

    Pool pool;
    MambaW m = make_mamba(pool, mc);
    if (mc.flags & HSPEC_W_DS_PACKED) {
      const int dS = mc.H * mc.P * mc.N;
      const size_t pb = hspec_pack_w_ds_bytes(dS, mc.r);
      void* packed = pool.get(pb > 0 ? pb : 256);
      const long before = stub_launches();
      std::snprintf(what, sizeof what, "random %d: pack_w_ds", i);
      const hspec_status st = hspec_pack_w_ds(dS, mc.r, m.w.W_dS, packed, nullptr);
      accepted_or_refused(what, st, before);
      if (st == HSPEC_OK) m.w.W_dS = packed;
      else mc.flags &= ~HSPEC_W_DS_PACKED;
    }
    const hspec_attn_w aw = make_attn(pool, ac);
    const Paged pg = make_paged(pool, ac);
    const size_t s = esz(dt), M = (size_t)B * mc.k, dm = (size_t)mc.d_model;
    const float* n1 = (const float*)pool.get(dm * 4);
    const float* n2 = (const float*)pool.get(dm * 4);
    void* h = pool.get((size_t)B * mc.d_h * s);
    void* e = pool.get(M * dm * s);
    float* out = (float*)pool.get(M * dm * 4);
    {
      const size_t n = hspec_draft_step_workspace(&mc, &ac, max_ctx);
      void* ws = random_ws(pool, n);
      const long before = stub_launches();
      std::snprintf(what, sizeof what, "random %d: draft_step", i);
      accepted_or_refused(what, hspec_draft_step(&mc, &m.w, n1, &ac, &aw, n2, h, e, pg.kc, pg.vc, pg.pt, pg.lens,
                                                 max_ctx, out, ws, n > 0 ? n : 256, nullptr),
                          before);
    }
    {
      const size_t n = hspec_mamba_block_scan_workspace(&mc);
      void* ws = random_ws(pool, n);
      float* S = (float*)pool.get((size_t)B * mc.H * mc.P * mc.N * 4);
      const long before = stub_launches();
      std::snprintf(what, sizeof what, "random %d: mamba_block_scan", i);
      accepted_or_refused(what, hspec_mamba_block_scan(&mc, &m.w, h, e, out, r(2) ? S : nullptr, ws, n > 0 ? n : 256,
                                                       nullptr),
                          before);
    }
    {
      const size_t n = hspec_target_kv_block_attn_workspace(&ac, max_ctx);
      void* ws = random_ws(pool, n);
      const long before = stub_launches();
      std::snprintf(what, sizeof what, "random %d: target_kv_block_attn", i);
      accepted_or_refused(what, hspec_target_kv_block_attn(&ac, &aw, e, pg.kc, pg.vc, pg.pt, pg.lens, max_ctx, out, ws,
                                                           n > 0 ? n : 256, nullptr),
                          before);
    }
  }
  std::printf("ok   random configurations: %d calls accepted, %d refused\n", g_rand_ok, g_rand_rejected);
}

int main() {
  const hspec_dtype dts[2] = {HSPEC_BF16, HSPEC_F32};
  for (hspec_dtype dt : dts) {
    const char* tag = dt == HSPEC_BF16 ? "bf16" : "f32";
    char name[64];
    hspec_attn_cfg a = attn_cfg(dt, 3, 4, 256, 8, 2, 128);
    std::snprintf(name, sizeof name, "%s plain", tag);
    run_attention_calls(name, a, 100);
    std::snprintf(name, sizeof name, "%s empty contexts", tag);
    run_attention_calls(name, a, 0);
    hspec_attn_cfg w = attn_cfg(dt, 3, 4, 128, 4, 4, 64);
    w.window = 32; w.flags = HSPEC_BLOCK_CAUSAL; w.split_tokens = 64;
    std::snprintf(name, sizeof name, "%s window, causal, split 64", tag);
    run_attention_calls(name, w, 128);
    hspec_attn_cfg p = a;
    p.flags = HSPEC_ATTN_PRECISE_IO;
    std::snprintf(name, sizeof name, "%s precise I/O", tag);
    run_attention_calls(name, p, 100);
    hspec_attn_cfg sub = a;
    static const int32_t heads[2] = {3, 1};
    sub.Hkv_cache = 4; sub.kv_heads = heads;
    std::snprintf(name, sizeof name, "%s KV-head subset", tag);
    run_attention_calls(name, sub, 100);
    hspec_attn_cfg many = attn_cfg(dt, 600, 2, 64, 4, 1, 64);
    many.max_pages = 2; many.num_pages = 64;
    std::snprintf(name, sizeof name, "%s 600 requests (work list in its own launch)", tag);
    run_attention_calls(name, many, 20);

    hspec_mamba_cfg m = mamba_cfg(dt, 3, 4, 256, dt == HSPEC_BF16 ? 64 : 16);
    std::snprintf(name, sizeof name, "%s mamba", tag);
    run_mamba_calls(name, m);
    if (dt == HSPEC_BF16) {
      hspec_mamba_cfg pk = m;
      pk.flags = HSPEC_W_DS_PACKED;
      run_mamba_calls("bf16 mamba, packed W_dS", pk);
      run_step_calls("bf16 step, packed W_dS", pk, a, 100);
    }
    std::snprintf(name, sizeof name, "%s step", tag);
    run_step_calls(name, m, a, 100);
    std::snprintf(name, sizeof name, "%s step, KV-head subset", tag);
    run_step_calls(name, m, sub, 100);
    std::snprintf(name, sizeof name, "%s kv_inject", tag);
    run_inject_calls(name, a);
  }
  run_head_calls();
  run_queries();
  run_random_calls(300);
  std::printf("host sanitizer driver: %d cases passed\n", g_cases);
  return 0;
}
