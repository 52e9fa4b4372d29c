// Host stand-ins for the kernel launchers of kernels.h and the three HIP runtime calls the C ABI
// makes, so that abi.cpp (argument checks, workspace layout, launch sequence) can be built and
// run on the CPU under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Every "device" buffer of the driver is plain host memory registered with stub_register().
// Each launcher works out, from its arguments alone, the byte range of every buffer the real
// kernel reads or writes (the extents stated for each launcher in kernels.h), checks that the
// range lies inside one registered buffer (else it prints the launcher, the argument and the
// range, and aborts), then reads the range (inputs) or fills it (outputs), so that the
// sanitizer also sees every access.  Launches are counted, so the driver can check that a
// rejected call enqueued nothing.
//
// gemm_scratch_elems, gemm_f16_out_ok and attention_sweep_grid depend on the GPU kernels'
// tile plans and occupancy; they are stood in for here by functions of the same contract
// (split-K scratch of ksplit * M * N elements; fp16 output on the weight-streaming shapes;
// a persistent grid of 512 workgroups).
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "stub_registry.h"

namespace {

struct Region {
  const char* base;
  size_t bytes;
};
std::vector<Region>& regions() {
  static std::vector<Region> r;
  return r;
}
long g_launches = 0;
const char* g_where = "";

[[noreturn]] void die(const char* what, const void* p, size_t bytes) {
  std::fprintf(stderr, "stub: %s: %s [%p, +%zu) is outside every registered buffer\n", g_where, what, p, bytes);
  std::fflush(stderr);
  std::abort();
}

// Regions that abi.cpp cut from the workspace of the current calls (hspec_host_carve).
std::vector<Region>& carves() {
  static std::vector<Region> r;
  return r;
}

bool inside(const Region& r, const char* c, size_t bytes) {
  return c >= r.base && bytes <= r.bytes && (size_t)(c - r.base) <= r.bytes - bytes;
}

// An access [p, p + bytes) must lie inside one registered buffer and, when it starts in a
// region cut from a workspace, inside that region: a region cut too small for what the kernel
// touches spills into its neighbour, which stays inside the workspace.
void check(const char* what, const void* p, size_t bytes) {
  if (!p) {
    std::fprintf(stderr, "stub: %s: %s is NULL\n", g_where, what);
    std::abort();
  }
  const char* c = static_cast<const char*>(p);
  for (const Region& r : carves())
    if (c >= r.base && c < r.base + r.bytes) {
      if (inside(r, c, bytes)) return;
      std::fprintf(stderr, "stub: %s: %s [%p, +%zu) spills out of its workspace region [%p, +%zu)\n", g_where, what,
                   p, bytes, (const void*)r.base, r.bytes);
      std::abort();
    }
  for (const Region& r : regions())
    if (inside(r, c, bytes)) return;
  die(what, p, bytes);
}

// An input: its whole extent is read.
volatile unsigned char g_sink;
void rd(const char* what, const void* p, size_t bytes) {
  check(what, p, bytes);
  const unsigned char* c = static_cast<const unsigned char*>(p);
  unsigned char x = 0;
  for (size_t i = 0; i < bytes; i += 61) x ^= c[i];
  if (bytes) x ^= c[bytes - 1];
  g_sink = x;
}
void rd_opt(const char* what, const void* p, size_t bytes) {
  if (p) rd(what, p, bytes);
}
// An output: its whole extent is written.
void wr(const char* what, void* p, size_t bytes) {
  check(what, p, bytes);
  std::memset(p, 0, bytes);
}
void wr_opt(const char* what, void* p, size_t bytes) {
  if (p) wr(what, p, bytes);
}
// Elements of a row-major matrix of `rows` rows of `cols` with leading dimension ld.
size_t strided(int rows, int cols, int ld) { return rows <= 0 ? 0 : (size_t)(rows - 1) * ld + cols; }

struct Scope {
  explicit Scope(const char* w) { g_where = w; ++g_launches; }
};

constexpr size_t BF = sizeof(hspec::bf16), F = sizeof(float), I = sizeof(int32_t);

}  // namespace

void stub_register(const void* p, size_t bytes) { regions().push_back({static_cast<const char*>(p), bytes}); }
void stub_unregister(const void* p) {
  auto& r = regions();
  for (size_t i = 0; i < r.size(); ++i)
    if (r[i].base == p) {
      auto& v = carves();   // the workspace regions cut from a freed buffer go with it
      for (size_t j = v.size(); j-- > 0;)
        if (v[j].base >= r[i].base && v[j].base < r[i].base + r[i].bytes) v.erase(v.begin() + (long)j);
      r.erase(r.begin() + (long)i);
      return;
    }
}
long stub_launches() { return g_launches; }

// A new region replaces every region of an earlier call that it overlaps.
void hspec_host_carve(const void* p, size_t bytes) {
  const char* c = static_cast<const char*>(p);
  auto& v = carves();
  for (size_t i = v.size(); i-- > 0;)
    if (v[i].bytes == 0 || (c < v[i].base + v[i].bytes && v[i].base < c + bytes)) v.erase(v.begin() + (long)i);
  if (bytes) v.push_back({c, bytes});
}

namespace hspec {

bool gemm_f16_out_ok(int M, int N, int K) { return M > 0 && M <= 128 && K % 32 == 0 && N % 4 == 0; }

size_t gemm_scratch_elems(int M, int N, int K, bool, bool) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  return K >= 512 ? (size_t)4 * M * N : 0;
}

int attention_sweep_grid(int D, int R, bool) { return (D == 64 || D == 128) && R >= 1 && R <= 128 ? 512 : 0; }

hipError_t launch_gemm(const GemmArgs& g, hipStream_t) {
  Scope s("launch_gemm");
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.lda < g.K || g.ldw < g.K) die("lda/ldw below K", nullptr, 0);
  rd("A_hi", g.A_hi, strided(g.M, g.K, g.lda) * BF);
  rd_opt("A_lo", g.A_lo, strided(g.M, g.K, g.lda) * BF);
  if (g.w_packed) {
    rd("W_hi (packed)", g.W_hi, (size_t)g.N * g.K * BF);
  } else if (g.W2) {
    const int n3 = g.N - g.N1 - g.N2;
    if (g.N1 <= 0 || g.N2 <= 0 || n3 < 0 || (n3 > 0) != (g.W3 != nullptr)) die("W segments", nullptr, 0);
    rd("W_hi", g.W_hi, strided(g.N1, g.K, g.ldw) * BF);
    rd("W2", g.W2, strided(g.N2, g.K, g.ldw) * BF);
    if (n3) rd("W3", g.W3, strided(n3, g.K, g.ldw) * BF);
  } else {
    rd("W_hi", g.W_hi, strided(g.N, g.K, g.ldw) * BF);
    rd_opt("W_lo", g.W_lo, strided(g.N, g.K, g.ldw) * BF);
  }
  if (g.R) {
    if (g.ldr < g.N) die("ldr below N", g.R, 0);
    rd("R", g.R, strided(g.M, g.N, g.ldr) * (g.r_bf16 ? BF : F));
  }
  if (!g.C && !g.C_hi && !g.C_h16) die("no output", nullptr, 0);
  if (g.C) {
    if (g.ldc < g.N) die("ldc below N", g.C, 0);
    wr("C", g.C, strided(g.M, g.N, g.ldc) * F);
  }
  if (g.f16 && !g.w_packed) die("fp16 operands without the packed W", nullptr, 0);
  if (g.C_hi || g.C_lo || g.C_h16) {
    if (g.ldch < g.N) die("ldch below N", g.C_hi, 0);
    wr_opt("C_hi", g.C_hi, strided(g.M, g.N, g.ldch) * BF);
    wr_opt("C_lo", g.C_lo, strided(g.M, g.N, g.ldch) * BF);
    if (g.C_h16 && !gemm_f16_out_ok(g.M, g.N, g.K)) return hipErrorInvalidValue;
    wr_opt("C_h16", g.C_h16, strided(g.M, g.N, g.ldch) * sizeof(_Float16));
    if (g.C_l16 && !g.C_h16) die("C_l16 without C_h16", g.C_l16, 0);
    wr_opt("C_l16", g.C_l16, strided(g.M, g.N, g.ldch) * sizeof(_Float16));
  }
  const size_t need = gemm_scratch_elems(g.M, g.N, g.K, g.A_lo != nullptr, g.W_lo != nullptr);
  if (need && g.part_cap >= need) wr("part", g.part, need * F);
  return hipSuccess;
}

hipError_t launch_pack_w(const bf16* W, int N, int K, _Float16* Wp, hipStream_t) {
  Scope s("launch_pack_w");
  rd("W", W, (size_t)N * K * BF);
  wr("Wp", Wp, (size_t)N * K * BF);
  return hipSuccess;
}

namespace {
void plan_extents(const AttnArgs& a, int clear_words) {
  rd("ctx_lens", a.ctx_lens, (size_t)a.B * I);
  wr_opt("status (cleared)", a.status, (size_t)clear_words * I);
  if (clear_words > 0 && !a.status) die("status", nullptr, 0);
  wr("units", a.units, (size_t)4 * a.B * a.max_splits * I);
  wr("req", a.req, (size_t)2 * a.B * I);
  wr("status[0, 3)", a.status, 3 * I);
}
}  // namespace

hipError_t launch_attention_plan(const AttnArgs& a, int clear_words, hipStream_t) {
  Scope s("launch_attention_plan");
  plan_extents(a, clear_words);
  return hipSuccess;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t, unsigned parts) {
  Scope s("launch_attention");
  const int R = a.T * (a.Hq / a.Hkv);
  const size_t q = (size_t)a.B * a.T * a.Hq * a.D, kv = (size_t)a.B * a.T * a.Hkv * a.D;
  const size_t cache = (size_t)a.num_pages * a.ps * a.Hkv_cache * a.D;
  const size_t items = (size_t)a.B * a.Hkv * a.max_splits;
  if (a.Hkv_cache < a.Hkv) die("Hkv_cache below Hkv", nullptr, 0);
  rd("q_hi", a.q_hi, q * BF);
  rd_opt("q_lo", a.q_lo, q * BF);
  rd("kb_hi", a.kb_hi, kv * BF);
  rd_opt("kb_lo", a.kb_lo, kv * BF);
  rd("vb_hi", a.vb_hi, kv * BF);
  rd_opt("vb_lo", a.vb_lo, kv * BF);
  rd("page_table", a.page_table, (size_t)a.B * a.max_pages * I);
  rd("ctx_lens", a.ctx_lens, (size_t)a.B * I);
  rd("units", a.units, (size_t)4 * a.B * a.max_splits * I);
  rd("req", a.req, (size_t)2 * a.B * I);
  wr("status", a.status, 3 * I);
  if (parts & ATTN_SWEEP) {
    rd("kc_hi", a.kc_hi, cache * BF);
    rd_opt("kc_lo", a.kc_lo, cache * BF);
    rd("vc_hi", a.vc_hi, cache * BF);
    rd_opt("vc_lo", a.vc_lo, cache * BF);
    // a single split per request without the precise path writes o directly
    if (a.max_splits > 1 || !a.block_in_sweep) {
      wr("part_o", a.part_o, items * R * a.D * F);
      wr("part_ml", a.part_ml, items * R * 2 * F);
    }
  }
  if (parts & ATTN_REDUCE) {
    if (a.part_o) rd("part_o", a.part_o, items * R * a.D * F);
    if (a.part_ml) rd("part_ml", a.part_ml, items * R * 2 * F);
  }
  if (!a.o_f32 && !a.o_bf16) die("no output", nullptr, 0);
  wr_opt("o_f32", a.o_f32, q * F);
  wr_opt("o_bf16", a.o_bf16, q * BF);
  wr_opt("o_bf16_lo", a.o_bf16_lo, q * BF);
  return hipSuccess;
}

hipError_t launch_gather_slots(int B, int max_pages, int, int, const int32_t* page_table, const int32_t* ctx_lens,
                               int max_ctx_len, int32_t* slots, int* status, hipStream_t) {
  Scope s("launch_gather_slots");
  rd("page_table", page_table, (size_t)B * max_pages * I);
  rd("ctx_lens", ctx_lens, (size_t)B * I);
  if (max_ctx_len > 0) wr("slots", slots, (size_t)B * max_ctx_len * I);
  wr_opt("status", status, I);
  return hipSuccess;
}

hipError_t launch_ssd_scan(const ScanArgs& a, hipStream_t) {
  Scope s("launch_ssd_scan");
  const int rows = a.B * a.T;
  const size_t st = (size_t)a.B * a.H * a.P * a.N;
  if (a.x_ld < a.H * a.P || a.bc_ld < a.G * a.N || a.dt_ld < a.H) die("leading dimension", nullptr, 0);
  rd("x_hi", a.x_hi, strided(rows, a.H * a.P, a.x_ld) * BF);
  rd_opt("x_lo", a.x_lo, strided(rows, a.H * a.P, a.x_ld) * BF);
  rd("dt", a.dt, strided(rows, a.H, a.dt_ld) * F);
  rd("A", a.A, (size_t)a.H * F);
  rd("B_hi", a.B_hi, strided(rows, a.G * a.N, a.bc_ld) * BF);
  rd_opt("B_lo", a.B_lo, strided(rows, a.G * a.N, a.bc_ld) * BF);
  rd("C_hi", a.C_hi, strided(rows, a.G * a.N, a.bc_ld) * BF);
  rd_opt("C_lo", a.C_lo, strided(rows, a.G * a.N, a.bc_ld) * BF);
  rd("Dskip", a.Dskip, (size_t)a.H * F);
  if (a.S0_h16 && (a.S0_hi || a.S0_lo)) die("S0 given both as fp16 and as bf16 planes", a.S0_h16, 0);
  rd_opt("S0_hi", a.S0_hi, st * BF);
  rd_opt("S0_lo", a.S0_lo, st * BF);
  rd_opt("S0_h16", a.S0_h16, st * sizeof(_Float16));
  wr("y", a.y, (size_t)rows * a.H * a.P * F);
  wr_opt("S_final", a.S_final, st * F);
  return hipSuccess;
}

hipError_t launch_rmsnorm_planes(const void* x, int x_bf16, const float* w, int rows, int n, float, bf16* out_hi,
                                 bf16* out_lo, hipStream_t) {
  Scope s("launch_rmsnorm_planes");
  rd("x", x, (size_t)rows * n * (x_bf16 ? BF : F));
  rd("w", w, (size_t)n * F);
  wr("out_hi", out_hi, (size_t)rows * n * BF);
  wr_opt("out_lo", out_lo, (size_t)rows * n * BF);
  return hipSuccess;
}

hipError_t launch_conv_split(const ConvArgs& a, hipStream_t) {
  Scope s("launch_conv_split");
  const size_t rows = (size_t)a.B * a.T, di = (size_t)a.H * a.P, gn = (size_t)a.G * a.N;
  const size_t conv_dim = di + 2 * gn, dproj = 2 * di + 2 * gn + a.H;
  rd("zxbcdt", a.zxbcdt, rows * dproj * F);
  rd("conv_w", a.conv_w, conv_dim * a.K * (a.w_bf16 ? BF : F));
  rd("conv_b", a.conv_b, conv_dim * (a.w_bf16 ? BF : F));
  rd("dt_bias", a.dt_bias, (size_t)a.H * F);
  wr("x_hi", a.x_hi, rows * di * BF);
  wr_opt("x_lo", a.x_lo, rows * di * BF);
  wr("B_hi", a.B_hi, rows * gn * BF);
  wr_opt("B_lo", a.B_lo, rows * gn * BF);
  wr("C_hi", a.C_hi, rows * gn * BF);
  wr_opt("C_lo", a.C_lo, rows * gn * BF);
  wr("dt", a.dt, rows * a.H * F);
  return hipSuccess;
}

hipError_t launch_gated_rmsnorm(const float* y, const float* z, int z_ld, const float* w, int rows, int n, int,
                                float, bf16* out_hi, bf16* out_lo, hipStream_t) {
  Scope s("launch_gated_rmsnorm");
  if (z_ld < n) die("z_ld below n", z, 0);
  rd("y", y, (size_t)rows * n * F);
  rd("z", z, strided(rows, n, z_ld) * F);
  rd("w", w, (size_t)n * F);
  wr("out_hi", out_hi, (size_t)rows * n * BF);
  wr_opt("out_lo", out_lo, (size_t)rows * n * BF);
  return hipSuccess;
}

hipError_t launch_qk_norm_rope(const float* qkv, const float* qw, const float* kw, const int32_t* ctx_lens, int B,
                               int T, int Hq, int Hkv, int D, float, double, bf16* q_hi, bf16* q_lo, bf16* k_hi,
                               bf16* k_lo, bf16* v_hi, bf16* v_lo, hipStream_t, const AttnArgs* plan,
                               int plan_clear) {
  Scope s("launch_qk_norm_rope");
  const size_t rows = (size_t)B * T;
  rd("qkv", qkv, rows * (Hq + 2 * Hkv) * D * F);
  if (Hq > 0) {
    rd("qw", qw, (size_t)D * F);
    wr("q_hi", q_hi, rows * Hq * D * BF);
    wr_opt("q_lo", q_lo, rows * Hq * D * BF);
  }
  rd("kw", kw, (size_t)D * F);
  rd("ctx_lens", ctx_lens, (size_t)B * I);
  wr("k_hi", k_hi, rows * Hkv * D * BF);
  wr_opt("k_lo", k_lo, rows * Hkv * D * BF);
  wr("v_hi", v_hi, rows * Hkv * D * BF);
  wr_opt("v_lo", v_lo, rows * Hkv * D * BF);
  if (plan) {
    if (plan->B > kWorklistFusedMax) die("fused work list above kWorklistFusedMax requests", nullptr, 0);
    plan_extents(*plan, plan_clear);
  }
  return hipSuccess;
}

hipError_t launch_split_planes(const float* x, size_t n, bf16* hi, bf16* lo, hipStream_t) {
  Scope s("launch_split_planes");
  rd("x", x, n * F);
  wr("hi", hi, n * BF);
  wr_opt("lo", lo, n * BF);
  return hipSuccess;
}

hipError_t launch_silu_mul(const float* gu, int rows, int ff, bf16* hi, bf16* lo, hipStream_t) {
  Scope s("launch_silu_mul");
  rd("gu", gu, (size_t)rows * 2 * ff * F);
  wr("hi", hi, (size_t)rows * ff * BF);
  wr_opt("lo", lo, (size_t)rows * ff * BF);
  return hipSuccess;
}

hipError_t launch_kv_append(const bf16* k_hi, const bf16* k_lo, const bf16* v_hi, const bf16* v_lo, int B, int n,
                            int Hkv, int D, const int32_t* page_table, int max_pages, int num_pages, int ps,
                            const int32_t* ctx_lens, void* k_cache, void* v_cache, int cache_bf16, int* status,
                            hipStream_t) {
  Scope s("launch_kv_append");
  const size_t rows = (size_t)B * n * Hkv * D, cache = (size_t)num_pages * ps * Hkv * D * (cache_bf16 ? BF : F);
  rd("k_hi", k_hi, rows * BF);
  rd_opt("k_lo", k_lo, rows * BF);
  rd("v_hi", v_hi, rows * BF);
  rd_opt("v_lo", v_lo, rows * BF);
  rd("page_table", page_table, (size_t)B * max_pages * I);
  rd("ctx_lens", ctx_lens, (size_t)B * I);
  wr("k_cache", k_cache, cache);
  wr("v_cache", v_cache, cache);
  wr("status", status, I);
  return hipSuccess;
}

hipError_t launch_zero_words(int* p, int n, hipStream_t) {
  Scope s("launch_zero_words");
  wr("words", p, (size_t)n * I);
  return hipSuccess;
}

hipError_t launch_head_clear(const HeadArgs& a, int status_words, hipStream_t) {
  Scope s("launch_head_clear");
  wr("status", a.status, (size_t)status_words * I);
  wr("keys", a.keys, (size_t)a.B * a.k * sizeof(unsigned long long));
  return hipSuccess;
}

hipError_t launch_markov_head(const HeadArgs& a, hipStream_t) {
  Scope s("launch_markov_head");
  const size_t M = (size_t)a.B * a.k, VR = (size_t)a.V * a.R;
  rd("E", a.E, VR * BF);
  rd("U", a.U, VR * BF);
  rd("base", a.base, M * a.V * F);
  rd_opt("gumbel", a.gumbel, M * a.V * F);
  rd("prev", a.prev, (size_t)a.B * I);
  rd_opt("forced", a.forced, M * I);
  wr_opt("logits", a.logits, M * a.V * F);
  wr("keys", a.keys, M * sizeof(unsigned long long));
  wr("tokens", a.tokens, M * I);
  wr("status", a.status, I);
  return hipSuccess;
}

}  // namespace hspec

// The HIP runtime calls abi.cpp makes itself.
extern "C" hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t) {
  Scope s("hipMemcpyAsync");
  if (kind == hipMemcpyDeviceToHost || kind == hipMemcpyDeviceToDevice) rd("src", src, bytes);
  if (kind == hipMemcpyHostToDevice || kind == hipMemcpyDeviceToDevice) wr("dst", dst, bytes);
  std::memcpy(dst, src, bytes);   // host memory on the other side: the sanitizer checks it
  return hipSuccess;
}
extern "C" hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
extern "C" const char* hipGetErrorString(hipError_t) { return "stub error"; }
