// C ABI of the drafting step: argument validation, workspace layout, and the stream-ordered
// launch sequence of each entry point.  Host code only; every kernel lives in a .hip file.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <initializer_list>
#include <cstdio>

#include "hspec.h"
#include "kernels.h"

#define HSPEC_API extern "C" __attribute__((visibility("default")))

using hspec::bf16;

namespace {

// Message of the last failing call on this thread.  A plain array: nothing in the library
// runs a destructor at thread or process exit.
thread_local char g_err[512];

void clear_err() { g_err[0] = 0; }

hspec_status fail(hspec_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(HSPEC_ERR_LAUNCH, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr size_t ALIGN = 256;

#ifdef HSPEC_HOST_SANITIZE
}  // namespace
// Host sanitizer build only: told every region cut from a caller's workspace.
void hspec_host_carve(const void* p, size_t bytes);
namespace {
#endif

// Bump allocator over the caller's workspace.  With base == nullptr it only measures.
struct Arena {
  char* base = nullptr;
  size_t off = 0;
  template <class T>
  T* take(size_t count) {
    size_t o = (off + ALIGN - 1) / ALIGN * ALIGN;
    off = o + count * sizeof(T);
#ifdef HSPEC_HOST_SANITIZE
    if (base) hspec_host_carve(base + o, count * sizeof(T));
#endif
    return base ? reinterpret_cast<T*>(base + o) : nullptr;
  }
  size_t size() const { return (off + ALIGN - 1) / ALIGN * ALIGN; }
};

bool is_f32(hspec_dtype d) { return d == HSPEC_F32; }
long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }
bool dtype_ok(hspec_dtype d) { return d == HSPEC_BF16 || d == HSPEC_F32; }

// A storage-dtype matrix as MFMA planes: bf16 storage is its own hi plane; fp32 storage is
// split into (hi, lo) inside the workspace.
struct Planes {
  const bf16* hi = nullptr;
  const bf16* lo = nullptr;
};
struct SplitSlot {
  bf16* hi = nullptr;
  bf16* lo = nullptr;
  size_t n = 0;
};
SplitSlot reserve_split(Arena& ar, hspec_dtype d, size_t n) {
  SplitSlot s;
  if (is_f32(d)) {
    s.hi = ar.take<bf16>(n);
    s.lo = ar.take<bf16>(n);
    s.n = n;
  }
  return s;
}
hipError_t as_planes(const void* src, hspec_dtype d, const SplitSlot& slot, Planes& out, hipStream_t st) {
  if (!is_f32(d)) {
    out.hi = static_cast<const bf16*>(src);
    out.lo = nullptr;
    return hipSuccess;
  }
  out.hi = slot.hi;
  out.lo = slot.lo;
  return hspec::launch_split_planes(static_cast<const float*>(src), slot.n, slot.hi, slot.lo, st);
}

// The planes as_planes gave for src on an earlier call with the same workspace, without
// splitting again: src itself for bf16 storage, the workspace slot for fp32.
Planes planes_in_place(const void* src, hspec_dtype d, const SplitSlot& slot) {
  if (!is_f32(d)) return Planes{static_cast<const bf16*>(src), nullptr};
  return Planes{slot.hi, slot.lo};
}

// Split-K scratch shared by a sequence of GEMMs on one stream, sized for the largest.
struct GemmScratch {
  float* p = nullptr;
  size_t cap = 0;
};
GemmScratch reserve_gemm(Arena& ar, hspec_dtype d, std::initializer_list<std::array<int, 3>> mnk) {
  GemmScratch s;
  for (const auto& x : mnk) s.cap = std::max(s.cap, hspec::gemm_scratch_elems(x[0], x[1], x[2], true, is_f32(d)));
  if (s.cap) s.p = ar.take<float>(s.cap);
  return s;
}
void use_scratch(hspec::GemmArgs& g, const GemmScratch& s) {
  g.part = s.p;
  g.part_cap = s.cap;
}

// ------------------------------------------------------------------------- validation

hspec_status check_mamba(const hspec_mamba_cfg* c, const hspec_mamba_w* w, bool full) {
  if (!c || !w) return fail(HSPEC_ERR_NULL, "mamba config or weights is NULL");
  if (!dtype_ok(c->dtype)) return fail(HSPEC_ERR_DTYPE, "unknown dtype %d", (int)c->dtype);
  if (c->B <= 0 || c->d_h <= 0 || c->r <= 0 || c->H <= 0 || c->P <= 0 || c->N <= 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive mamba dimension");
  if (c->P != 64) return fail(HSPEC_ERR_UNSUPPORTED, "P (head dim) must be 64, got %d", c->P);
  if (c->N != 16 && c->N != 32 && c->N != 64 && c->N != 128)
    return fail(HSPEC_ERR_UNSUPPORTED, "N (d_state) must be 16, 32, 64 or 128, got %d", c->N);
  if (c->d_h % 8 || c->r % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_h and r must be multiples of 8");
  if (c->flags & ~(unsigned)(HSPEC_W_DS_PACKED | HSPEC_MAMBA_PRECISE_IO))
    return fail(HSPEC_ERR_UNSUPPORTED, "unknown mamba flags 0x%x", c->flags);
  if ((c->flags & HSPEC_W_DS_PACKED) && (is_f32(c->dtype) || c->r % 64 || c->d_h % 32))
    return fail(HSPEC_ERR_UNSUPPORTED, "a packed W_dS needs bf16 storage, r %% 64 == 0 and d_h %% 32 == 0");
  if (!w->W_r || !w->W_dS) return fail(HSPEC_ERR_NULL, "W_r or W_dS is NULL");
  if (!full) return HSPEC_OK;
  if (c->k <= 0 || c->d_model <= 0 || c->G <= 0 || c->chunk <= 0 || c->conv_w <= 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive mamba dimension");
  if (c->H % c->G) return fail(HSPEC_ERR_SHAPE, "H %% G != 0 (H=%d, G=%d)", c->H, c->G);
  if (c->chunk > 16) return fail(HSPEC_ERR_UNSUPPORTED, "chunk must be <= 16, got %d", c->chunk);
  if (c->conv_w > 8) return fail(HSPEC_ERR_UNSUPPORTED, "conv_w must be <= 8, got %d", c->conv_w);
  if (c->d_model % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_model must be a multiple of 8");
  if ((c->H * c->P) % c->G) return fail(HSPEC_ERR_SHAPE, "d_inner %% G != 0");
  if (!w->W_in || !w->conv_w || !w->conv_b || !w->dt_bias || !w->A_log || !w->D || !w->gnorm_w || !w->W_out)
    return fail(HSPEC_ERR_NULL, "a mamba weight pointer is NULL");
  return HSPEC_OK;
}

// KV heads per slot of the target cache.
int cache_heads(const hspec_attn_cfg& c) { return c.Hkv_cache > 0 ? c.Hkv_cache : c.Hkv; }

hspec_status check_attn_cfg(const hspec_attn_cfg* c, int max_ctx_len) {
  if (!c) return fail(HSPEC_ERR_NULL, "attention config is NULL");
  if (!dtype_ok(c->dtype)) return fail(HSPEC_ERR_DTYPE, "unknown dtype %d", (int)c->dtype);
  if (c->B <= 0 || c->k <= 0 || c->Hq <= 0 || c->Hkv <= 0 || c->D <= 0 || c->page_size <= 0 ||
      c->max_pages <= 0 || c->num_pages <= 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive attention dimension");
  if (c->Hq % c->Hkv) return fail(HSPEC_ERR_SHAPE, "Hq %% Hkv != 0 (Hq=%d, Hkv=%d)", c->Hq, c->Hkv);
  if (c->D != 64 && c->D != 128) return fail(HSPEC_ERR_UNSUPPORTED, "D must be 64 or 128, got %d", c->D);
  if (c->flags & ~(unsigned)(HSPEC_BLOCK_CAUSAL | HSPEC_ATTN_PRECISE_IO))
    return fail(HSPEC_ERR_UNSUPPORTED, "unknown attention flags 0x%x", c->flags);
  if (c->k * (c->Hq / c->Hkv) > 128)
    return fail(HSPEC_ERR_UNSUPPORTED, "k * Hq/Hkv must be <= 128, got %d", c->k * (c->Hq / c->Hkv));
  if (c->Hkv_cache != 0 && (c->Hkv_cache < c->Hkv))
    return fail(HSPEC_ERR_SHAPE, "Hkv_cache (%d) < Hkv (%d)", c->Hkv_cache, c->Hkv);
  if (cache_heads(*c) > 16 && (c->kv_heads || c->Hkv_cache != 0))
    return fail(HSPEC_ERR_UNSUPPORTED, "KV-head reuse supports at most 16 cache heads, got %d", cache_heads(*c));
  if (c->kv_heads)
    for (int i = 0; i < c->Hkv; ++i)
      if (c->kv_heads[i] < 0 || c->kv_heads[i] >= cache_heads(*c))
        return fail(HSPEC_ERR_SHAPE, "kv_heads[%d] = %d outside [0, %d)", i, c->kv_heads[i], cache_heads(*c));
  if (c->window < 0) return fail(HSPEC_ERR_SHAPE, "window < 0");
  if (c->window > 0 && c->k > c->window) return fail(HSPEC_ERR_SHAPE, "k > window");
  if (c->split_tokens < 0 || c->split_tokens % 64)
    return fail(HSPEC_ERR_SHAPE, "split_tokens must be a non-negative multiple of 64");
  if (max_ctx_len < 0) return fail(HSPEC_ERR_SHAPE, "max_ctx_len < 0");
  if (c->B > 32767) return fail(HSPEC_ERR_UNSUPPORTED, "B must be <= 32767");
  if (c->page_size < 16 || (c->page_size & (c->page_size - 1)))
    return fail(HSPEC_ERR_UNSUPPORTED, "page_size must be a power of two >= 16, got %d", c->page_size);
  if (c->split_tokens > hspec::kMaxSplit)
    return fail(HSPEC_ERR_UNSUPPORTED, "split_tokens must be <= %d", hspec::kMaxSplit);
  const int swept = hspec::attention_swept_len(max_ctx_len, c->window);
  const int split = c->split_tokens > 0 ? c->split_tokens : hspec::attention_default_split(c->B, c->Hkv, swept);
  if (swept > 0 && ceil_div(swept, split) > 256)
    return fail(HSPEC_ERR_UNSUPPORTED, "swept context / split_tokens gives more than 256 splits");
  if ((long long)c->B * c->Hkv * (swept > 0 ? ceil_div(swept, 64) : 1) > 0x7fffffffLL)
    return fail(HSPEC_ERR_UNSUPPORTED, "B x Hkv x swept context is too large for the work list");
  if (split > hspec::kMaxSplit)   // the sweep holds one split's page ids in a fixed LDS array
    return fail(HSPEC_ERR_UNSUPPORTED, "swept context of %d keys needs splits above %d keys (at most 256 x %d)",
                swept, hspec::kMaxSplit, hspec::kMaxSplit);
  return HSPEC_OK;
}

hspec_status check_attn_w(const hspec_attn_cfg* c, const hspec_attn_w* w) {
  if (!w) return fail(HSPEC_ERR_NULL, "attention weights is NULL");
  if (!w->W_q || !w->W_k || !w->W_v || !w->W_o || !w->q_norm_w || !w->k_norm_w)
    return fail(HSPEC_ERR_NULL, "an attention weight pointer is NULL");
  if (c->d_model <= 0 || c->d_model % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_model must be a positive multiple of 8");
  return HSPEC_OK;
}

hspec_status check_ws(void* ws, size_t have, size_t need) {
  if (!ws) return fail(HSPEC_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % ALIGN) return fail(HSPEC_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (have < need) return fail(HSPEC_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", have, need);
  return HSPEC_OK;
}

// ---------------------------------------------------------------------- layout + launch

// F enters Proj_dS with the packed (fp16) W_dS as fp16 planes of F x 2^-kFScaleLog2, which
// Proj_r writes directly: finite for |F| < 65504 x 64 (about 4e6), full fp16 precision down to
// |F| = 2^-8, and an absolute error under 2^-19 below that.
constexpr int kFScaleLog2 = 6;

struct StatePlan {
  SplitSlot h, wr, wds;
  GemmScratch gs;
  bf16 *F_hi = nullptr, *F_lo = nullptr;        // bf16 planes of F (unpacked W_dS)
  _Float16 *F_h16 = nullptr, *F_l16 = nullptr;  // fp16 planes of F (packed W_dS; l16 only precise)
  bf16 *S0_hi = nullptr, *S0_lo = nullptr;
  _Float16* S0_h16 = nullptr;
};

void plan_state(Arena& ar, const hspec_mamba_cfg& c, bool s0_planes, StatePlan& p) {
  const size_t dS = (size_t)c.H * c.P * c.N;
  p.h = reserve_split(ar, c.dtype, (size_t)c.B * c.d_h);
  p.wr = reserve_split(ar, c.dtype, (size_t)c.r * c.d_h);
  p.wds = reserve_split(ar, c.dtype, dS * c.r);
  if (c.flags & HSPEC_W_DS_PACKED) {
    // one fp16 plane (11 significant bits), or hi/lo fp16 planes with HSPEC_MAMBA_PRECISE_IO
    p.F_h16 = ar.take<_Float16>((size_t)c.B * c.r);
    if (c.flags & HSPEC_MAMBA_PRECISE_IO) p.F_l16 = ar.take<_Float16>((size_t)c.B * c.r);
  } else {
    p.F_hi = ar.take<bf16>((size_t)c.B * c.r);
    p.F_lo = ar.take<bf16>((size_t)c.B * c.r);
  }
  p.gs = reserve_gemm(ar, c.dtype, {{c.B, c.r, c.d_h}, {c.B, (int)dS, c.r}});
  if (s0_planes) {
    // S0 only feeds the scan: one fp16 plane (11 significant bits, half the bytes of hi/lo
    // bf16 planes) where the state projection runs on the weight-streaming path, else hi/lo
    if (!is_f32(c.dtype) && hspec::gemm_f16_out_ok(c.B, (int)dS, c.r)) {
      p.S0_h16 = ar.take<_Float16>((size_t)c.B * dS);
    } else {
      p.S0_hi = ar.take<bf16>((size_t)c.B * dS);
      p.S0_lo = ar.take<bf16>((size_t)c.B * dS);
    }
  }
}

// F = W_r h_last (bf16 planes, or fp16 planes for the packed W_dS), then S0 = W_dS F (fp32,
// bf16 planes and/or one fp16 plane).
hspec_status run_state(const hspec_mamba_cfg& c, const hspec_mamba_w& w, const void* h_last, const StatePlan& p,
                       float* S0_f32, hipStream_t st) {
  Planes h, wr, wds;
  HIP_TRY(as_planes(h_last, c.dtype, p.h, h, st));
  HIP_TRY(as_planes(w.W_r, c.dtype, p.wr, wr, st));
  HIP_TRY(as_planes(w.W_dS, c.dtype, p.wds, wds, st));
  hspec::GemmArgs g1;
  g1.A_hi = h.hi; g1.A_lo = h.lo; g1.lda = c.d_h;
  g1.W_hi = wr.hi; g1.W_lo = wr.lo; g1.ldw = c.d_h;
  g1.M = c.B; g1.N = c.r; g1.K = c.d_h;
  g1.C_hi = p.F_hi; g1.C_lo = p.F_lo; g1.ldch = c.r;
  g1.C_h16 = p.F_h16; g1.C_l16 = p.F_l16; g1.h16_scale = 1.f / (1 << kFScaleLog2);
  use_scratch(g1, p.gs);
  HIP_TRY(hspec::launch_gemm(g1, st));
  const int dS = c.H * c.P * c.N;
  hspec::GemmArgs g2;
  g2.A_hi = p.F_hi; g2.A_lo = p.F_lo; g2.lda = c.r;
  if (p.F_h16) {   // fp16 product with the packed W_dS (x 2^kPackScaleLog2), F x 2^-kFScaleLog2
    g2.A_hi = reinterpret_cast<const bf16*>(p.F_h16);
    g2.A_lo = reinterpret_cast<const bf16*>(p.F_l16);
    g2.f16 = 1;
    g2.out_scale = (float)(1 << kFScaleLog2) / (float)(1 << hspec::kPackScaleLog2);
  }
  g2.W_hi = wds.hi; g2.W_lo = wds.lo; g2.ldw = c.r;
  g2.M = c.B; g2.N = dS; g2.K = c.r;
  g2.C = S0_f32; g2.ldc = dS;
  g2.C_hi = p.S0_hi; g2.C_lo = p.S0_lo; g2.C_h16 = p.S0_h16; g2.ldch = dS;
  g2.w_packed = (c.flags & HSPEC_W_DS_PACKED) ? 1 : 0;
  use_scratch(g2, p.gs);
  HIP_TRY(hspec::launch_gemm(g2, st));
  return HSPEC_OK;
}

struct MambaPlan {
  StatePlan st;
  SplitSlot u_in, win, wout;
  bf16 *u_hi = nullptr, *u_lo = nullptr;      // normalised block input (draft step)
  float* zx = nullptr;
  bf16 *x_hi = nullptr, *x_lo = nullptr, *B_hi = nullptr, *B_lo = nullptr, *C_hi = nullptr, *C_lo = nullptr;
  float* dt = nullptr;
  float* y = nullptr;
  bf16 *yn_hi = nullptr, *yn_lo = nullptr;
  GemmScratch gs;
};

// Whether the Mamba projections take their activations as hi/lo planes (fp32 storage, or
// HSPEC_MAMBA_PRECISE_IO) or as one bf16 plane.
bool mamba_io_lo(const hspec_mamba_cfg& c) { return is_f32(c.dtype) || (c.flags & HSPEC_MAMBA_PRECISE_IO); }

void plan_mamba(Arena& ar, const hspec_mamba_cfg& c, bool u_norm, MambaPlan& p) {
  plan_state(ar, c, true, p.st);
  const size_t M = (size_t)c.B * c.k;
  const size_t di = (size_t)c.H * c.P, gn = (size_t)c.G * c.N;
  const size_t dproj = 2 * di + 2 * gn + c.H;
  const bool io_lo = mamba_io_lo(c);
  if (u_norm) {
    p.u_hi = ar.take<bf16>(M * c.d_model);
    if (io_lo) p.u_lo = ar.take<bf16>(M * c.d_model);
  } else {
    p.u_in = reserve_split(ar, c.dtype, M * c.d_model);
  }
  p.win = reserve_split(ar, c.dtype, dproj * c.d_model);
  p.wout = reserve_split(ar, c.dtype, (size_t)c.d_model * di);
  p.zx = ar.take<float>(M * dproj);
  p.x_hi = ar.take<bf16>(M * di);
  p.x_lo = ar.take<bf16>(M * di);   // x feeds the state update: kept as hi/lo planes
  p.B_hi = ar.take<bf16>(M * gn);
  p.B_lo = ar.take<bf16>(M * gn);
  p.C_hi = ar.take<bf16>(M * gn);
  p.C_lo = ar.take<bf16>(M * gn);
  p.dt = ar.take<float>(M * c.H);
  p.y = ar.take<float>(M * di);
  p.yn_hi = ar.take<bf16>(M * di);
  if (io_lo) p.yn_lo = ar.take<bf16>(M * di);
  p.gs = reserve_gemm(ar, c.dtype, {{(int)M, (int)dproj, c.d_model}, {(int)M, c.d_model, (int)di}});
}

// in_proj -> conv/split -> scan from S0 planes -> gated norm -> out_proj (+ residual R).
hspec_status run_mamba_core(const hspec_mamba_cfg& c, const hspec_mamba_w& w, Planes u, const MambaPlan& p,
                            const void* R, int r_bf16, float* out, float* S_final, hipStream_t st) {
  const int M = c.B * c.k;
  const int di = c.H * c.P, gn = c.G * c.N;
  const int dproj = 2 * di + 2 * gn + c.H;
  Planes win, wout;
  HIP_TRY(as_planes(w.W_in, c.dtype, p.win, win, st));
  HIP_TRY(as_planes(w.W_out, c.dtype, p.wout, wout, st));
  hspec::GemmArgs gi;
  gi.A_hi = u.hi; gi.A_lo = u.lo; gi.lda = c.d_model;
  gi.W_hi = win.hi; gi.W_lo = win.lo; gi.ldw = c.d_model;
  gi.M = M; gi.N = dproj; gi.K = c.d_model;
  gi.C = p.zx; gi.ldc = dproj;
  use_scratch(gi, p.gs);
  HIP_TRY(hspec::launch_gemm(gi, st));

  hspec::ConvArgs ca;
  ca.zxbcdt = p.zx; ca.conv_w = w.conv_w; ca.conv_b = w.conv_b; ca.w_bf16 = !is_f32(c.dtype);
  ca.dt_bias = w.dt_bias;
  ca.B = c.B; ca.T = c.k; ca.H = c.H; ca.P = c.P; ca.G = c.G; ca.N = c.N; ca.K = c.conv_w;
  ca.x_hi = p.x_hi; ca.x_lo = p.x_lo; ca.B_hi = p.B_hi; ca.B_lo = p.B_lo; ca.C_hi = p.C_hi; ca.C_lo = p.C_lo;
  ca.dt = p.dt;
  HIP_TRY(hspec::launch_conv_split(ca, st));

  hspec::ScanArgs sa;
  sa.x_hi = p.x_hi; sa.x_lo = p.x_lo; sa.dt = p.dt; sa.A = w.A_log; sa.A_is_log = 1;
  sa.B_hi = p.B_hi; sa.B_lo = p.B_lo; sa.C_hi = p.C_hi; sa.C_lo = p.C_lo; sa.Dskip = w.D;
  sa.S0_hi = p.st.S0_hi; sa.S0_lo = p.st.S0_lo; sa.S0_h16 = p.st.S0_h16; sa.y = p.y; sa.S_final = S_final;
  sa.B = c.B; sa.T = c.k; sa.H = c.H; sa.P = c.P; sa.N = c.N; sa.G = c.G; sa.chunk = c.chunk;
  sa.x_ld = di; sa.bc_ld = gn; sa.dt_ld = c.H;
  HIP_TRY(hspec::launch_ssd_scan(sa, st));

  HIP_TRY(hspec::launch_gated_rmsnorm(p.y, p.zx, dproj, w.gnorm_w, M, di, c.G, c.eps, p.yn_hi, p.yn_lo, st));

  hspec::GemmArgs go;
  go.A_hi = p.yn_hi; go.A_lo = p.yn_lo; go.lda = di;
  go.W_hi = wout.hi; go.W_lo = wout.lo; go.ldw = di;
  go.M = M; go.N = c.d_model; go.K = di;
  go.C = out; go.ldc = c.d_model;
  go.R = R; go.ldr = c.d_model; go.r_bf16 = r_bf16;
  use_scratch(go, p.gs);
  HIP_TRY(hspec::launch_gemm(go, st));
  return HSPEC_OK;
}

struct AttnPlan {
  SplitSlot x_in, wq, wk, wv, wo, kc, vc, qin, kbin, vbin;
  bf16 *xn_hi = nullptr, *xn_lo = nullptr;   // normalised input (draft step)
  float* qkv = nullptr;
  bf16 *q_hi = nullptr, *q_lo = nullptr, *k_hi = nullptr, *k_lo = nullptr, *v_hi = nullptr, *v_lo = nullptr;
  float* part_o = nullptr;
  float* part_ml = nullptr;
  int32_t* units = nullptr;
  int32_t* req = nullptr;
  bf16 *o_hi = nullptr, *o_lo = nullptr;
  int split = 0, max_splits = 0, auto_split = 0, min_split = 0;
  GemmScratch gs;
};

void plan_sweep(Arena& ar, const hspec_attn_cfg& c, int max_ctx_len, AttnPlan& p) {
  const int swept = hspec::attention_swept_len(max_ctx_len, c.window);
  p.split = c.split_tokens > 0 ? c.split_tokens : hspec::attention_default_split(c.B, c.Hkv, swept);
  // automatic splitting: the work-list kernel may cut requests finer than p.split (down to
  // attention_min_auto_split), so the buffers are sized for that many splits
  p.auto_split = c.split_tokens > 0 ? 0 : 1;
  p.min_split = p.auto_split ? hspec::attention_min_auto_split(p.split, swept) : p.split;
  // (a validated call has at most 256 splits; a query for any other config stays defined)
  const long long ns = swept > 0 ? ceil_div(swept, p.min_split) : 1;
  p.max_splits = (int)std::min<long long>(ns, INT_MAX);
  const int R = c.k * (c.Hq / c.Hkv);
  const size_t units = (size_t)c.B * c.Hkv * p.max_splits;
  p.units = ar.take<int32_t>((size_t)4 * c.B * p.max_splits);
  p.req = ar.take<int32_t>((size_t)2 * c.B);
  if (p.max_splits > 1 || (c.flags & HSPEC_ATTN_PRECISE_IO)) {   // split partials
    p.part_o = ar.take<float>(units * R * c.D);
    p.part_ml = ar.take<float>(units * R * 2);
  }
  const size_t cache = (size_t)c.num_pages * c.page_size * cache_heads(c) * c.D;
  p.kc = reserve_split(ar, c.dtype, cache);
  p.vc = reserve_split(ar, c.dtype, cache);
}

void plan_attn(Arena& ar, const hspec_attn_cfg& c, int max_ctx_len, bool x_norm, AttnPlan& p) {
  const size_t M = (size_t)c.B * c.k;
  const bool f32 = is_f32(c.dtype);
  const bool io_lo = f32 || (c.flags & HSPEC_ATTN_PRECISE_IO);   // hi/lo planes into W_q/k/v and W_o
  if (x_norm) {
    p.xn_hi = ar.take<bf16>(M * c.d_model);
    if (io_lo) p.xn_lo = ar.take<bf16>(M * c.d_model);
  } else {
    p.x_in = reserve_split(ar, c.dtype, M * c.d_model);
  }
  p.wq = reserve_split(ar, c.dtype, (size_t)c.Hq * c.D * c.d_model);
  p.wk = reserve_split(ar, c.dtype, (size_t)c.Hkv * c.D * c.d_model);
  p.wv = reserve_split(ar, c.dtype, (size_t)c.Hkv * c.D * c.d_model);
  p.wo = reserve_split(ar, c.dtype, (size_t)c.d_model * c.Hq * c.D);
  p.qkv = ar.take<float>(M * (c.Hq + 2 * c.Hkv) * c.D);
  // q, k and v: hi/lo planes for fp32 storage (the sweep's hi/lo products) and for precise
  // attention I/O (the reduction rebuilds the block keys in fp32 from both planes)
  p.q_hi = ar.take<bf16>(M * c.Hq * c.D);
  p.k_hi = ar.take<bf16>(M * c.Hkv * c.D);
  p.v_hi = ar.take<bf16>(M * c.Hkv * c.D);
  if (io_lo) {
    p.q_lo = ar.take<bf16>(M * c.Hq * c.D);
    p.k_lo = ar.take<bf16>(M * c.Hkv * c.D);
    p.v_lo = ar.take<bf16>(M * c.Hkv * c.D);
  }
  plan_sweep(ar, c, max_ctx_len, p);
  p.o_hi = ar.take<bf16>(M * c.Hq * c.D);
  if (io_lo) p.o_lo = ar.take<bf16>(M * c.Hq * c.D);
  // the fused QKV product (one launch over the three weight segments) and the separate ones
  p.gs = reserve_gemm(ar, c.dtype, {{(int)M, (c.Hq + 2 * c.Hkv) * c.D, c.d_model}, {(int)M, c.Hq * c.D, c.d_model},
                                    {(int)M, c.Hkv * c.D, c.d_model}, {(int)M, c.d_model, c.Hq * c.D}});
}

hspec::AttnArgs sweep_args(const hspec_attn_cfg& c, const AttnPlan& p, const int32_t* pt, const int32_t* lens,
                           int max_ctx_len, int* status) {
  hspec::AttnArgs a;
  a.page_table = pt; a.ctx_lens = lens;
  a.B = c.B; a.T = c.k; a.Hq = c.Hq; a.Hkv = c.Hkv; a.D = c.D; a.ps = c.page_size;
  a.Hkv_cache = cache_heads(c);
  a.kv_remap = c.kv_heads ? 1 : 0;   // (at most 16 cache heads then: checked)
  a.kv_map = 0;
  for (int h = 0; c.kv_heads && h < c.Hkv && h < 16; ++h) a.kv_map |= (unsigned long long)(c.kv_heads[h] & 15) << (4 * h);
  a.max_pages = c.max_pages; a.num_pages = c.num_pages; a.window = c.window;
  a.causal = (c.flags & HSPEC_BLOCK_CAUSAL) ? 1 : 0;
  a.block_in_sweep = (c.flags & HSPEC_ATTN_PRECISE_IO) ? 0 : 1;
  a.max_ctx_len = max_ctx_len; a.split = p.split; a.max_splits = p.max_splits;
  const float scale = c.scale > 0.f ? c.scale : 1.f / std::sqrt((float)c.D);
  a.scale_log2 = scale * 1.4426950408889634f;
  a.part_o = p.part_o; a.part_ml = p.part_ml; a.status = status; a.units = p.units; a.req = p.req;
  a.auto_split = p.auto_split; a.min_split = p.min_split;
  a.grid = a.auto_split ? hspec::attention_sweep_grid(c.D, c.k * (c.Hq / c.Hkv), is_f32(c.dtype)) : 0;
  return a;
}

// QKV projections -> q/k norm + RoPE -> sweep + reduce -> O projection (+ residual R).  The
// sweep's work list is built inside the q/k-norm + RoPE launch (its own launch, ahead of the
// projections, past kWorklistFusedMax requests), clearing the first plan_clear status words.
hspec_status run_attn_core(const hspec_attn_cfg& c, const hspec_attn_w& w, Planes xn, const void* k_cache,
                           const void* v_cache, const int32_t* pt, const int32_t* lens, int max_ctx_len,
                           const AttnPlan& p, const void* R, int r_bf16, float* out, int* status, int plan_clear,
                           hipStream_t st) {
  const int M = c.B * c.k;
  const hspec::AttnArgs plan = sweep_args(c, p, pt, lens, max_ctx_len, status);
  const bool plan_fused = c.B <= hspec::kWorklistFusedMax;
  if (!plan_fused) HIP_TRY(hspec::launch_attention_plan(plan, plan_clear, st));
  const int ldq = (c.Hq + 2 * c.Hkv) * c.D;
  Planes wq, wk, wv, wo, kc, vc;
  HIP_TRY(as_planes(w.W_q, c.dtype, p.wq, wq, st));
  HIP_TRY(as_planes(w.W_k, c.dtype, p.wk, wk, st));
  HIP_TRY(as_planes(w.W_v, c.dtype, p.wv, wv, st));
  HIP_TRY(as_planes(w.W_o, c.dtype, p.wo, wo, st));
  HIP_TRY(as_planes(k_cache, c.dtype, p.kc, kc, st));
  HIP_TRY(as_planes(v_cache, c.dtype, p.vc, vc, st));
  const Planes* ws[3] = {&wq, &wk, &wv};
  const int nrows[3] = {c.Hq * c.D, c.Hkv * c.D, c.Hkv * c.D};
  if (!wq.lo) {
    // one product over the three row segments [W_q; W_k; W_v]
    hspec::GemmArgs g;
    g.A_hi = xn.hi; g.A_lo = xn.lo; g.lda = c.d_model;
    g.W_hi = wq.hi; g.W2 = wk.hi; g.W3 = wv.hi; g.N1 = nrows[0]; g.N2 = nrows[1]; g.ldw = c.d_model;
    g.M = M; g.N = ldq; g.K = c.d_model;
    g.C = p.qkv; g.ldc = ldq;
    use_scratch(g, p.gs);
    HIP_TRY(hspec::launch_gemm(g, st));
  } else {
    int col = 0;
    for (int i = 0; i < 3; ++i) {
      hspec::GemmArgs g;
      g.A_hi = xn.hi; g.A_lo = xn.lo; g.lda = c.d_model;
      g.W_hi = ws[i]->hi; g.W_lo = ws[i]->lo; g.ldw = c.d_model;
      g.M = M; g.N = nrows[i]; g.K = c.d_model;
      g.C = p.qkv + col; g.ldc = ldq;
      use_scratch(g, p.gs);
      HIP_TRY(hspec::launch_gemm(g, st));
      col += nrows[i];
    }
  }
  HIP_TRY(hspec::launch_qk_norm_rope(p.qkv, w.q_norm_w, w.k_norm_w, lens, c.B, c.k, c.Hq, c.Hkv, c.D, c.eps,
                                     c.rope_theta, p.q_hi, p.q_lo, p.k_hi, p.k_lo, p.v_hi, p.v_lo, st,
                                     plan_fused ? &plan : nullptr, plan_clear));
  hspec::AttnArgs a = plan;
  a.q_hi = p.q_hi; a.q_lo = p.q_lo; a.kb_hi = p.k_hi; a.kb_lo = p.k_lo; a.vb_hi = p.v_hi; a.vb_lo = p.v_lo;
  a.kc_hi = kc.hi; a.kc_lo = kc.lo; a.vc_hi = vc.hi; a.vc_lo = vc.lo;
  a.o_bf16 = p.o_hi;
  a.o_bf16_lo = p.o_lo;
  HIP_TRY(hspec::launch_attention(a, st));
  hspec::GemmArgs g;
  g.A_hi = p.o_hi; g.A_lo = p.o_lo; g.lda = c.Hq * c.D;
  g.W_hi = wo.hi; g.W_lo = wo.lo; g.ldw = c.Hq * c.D;
  g.M = M; g.N = c.d_model; g.K = c.Hq * c.D;
  g.C = out; g.ldc = c.d_model;
  g.R = R; g.ldr = c.d_model; g.r_bf16 = r_bf16;
  use_scratch(g, p.gs);
  HIP_TRY(hspec::launch_gemm(g, st));
  return HSPEC_OK;
}

struct DraftPlan {
  MambaPlan m;
  float* x1 = nullptr;
  AttnPlan at;
};

void plan_draft(Arena& ar, const hspec_mamba_cfg& mc, const hspec_attn_cfg& ac, int max_ctx_len, DraftPlan& p) {
  plan_mamba(ar, mc, true, p.m);
  p.x1 = ar.take<float>((size_t)mc.B * mc.k * mc.d_model);
  plan_attn(ar, ac, max_ctx_len, true, p.at);
}

int* status_word(Arena& ar) { return ar.take<int>(ALIGN / sizeof(int)); }

}  // namespace

// ============================================================================ C ABI

HSPEC_API size_t hspec_state_init_workspace(const hspec_mamba_cfg* cfg) {
  if (!cfg) return 0;
  Arena ar;
  status_word(ar);
  StatePlan p;
  plan_state(ar, *cfg, false, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_state_init(const hspec_mamba_cfg* cfg, const hspec_mamba_w* w, const void* h_last,
                                        float* S0, void* workspace, size_t ws_bytes, void* stream) {
  clear_err();
  if (hspec_status s = check_mamba(cfg, w, false)) return s;
  if (!h_last || !S0) return fail(HSPEC_ERR_NULL, "h_last or S0 is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_state_init_workspace(cfg))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  StatePlan p;
  plan_state(ar, *cfg, false, p);
  HIP_TRY(hspec::launch_zero_words(status, hspec::kStatusClear, st));
  return run_state(*cfg, *w, h_last, p, S0, st);
}

HSPEC_API size_t hspec_mamba_block_scan_workspace(const hspec_mamba_cfg* cfg) {
  if (!cfg) return 0;
  Arena ar;
  status_word(ar);
  MambaPlan p;
  plan_mamba(ar, *cfg, false, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_mamba_block_scan(const hspec_mamba_cfg* cfg, const hspec_mamba_w* w,
                                              const void* h_last, const void* block_hidden, float* out,
                                              float* S_final, void* workspace, size_t ws_bytes, void* stream) {
  clear_err();
  if (hspec_status s = check_mamba(cfg, w, true)) return s;
  if (!h_last || !block_hidden || !out) return fail(HSPEC_ERR_NULL, "h_last, block_hidden or out is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_mamba_block_scan_workspace(cfg))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  MambaPlan p;
  plan_mamba(ar, *cfg, false, p);
  HIP_TRY(hspec::launch_zero_words(status, hspec::kStatusClear, st));
  if (hspec_status s = run_state(*cfg, *w, h_last, p.st, nullptr, st)) return s;
  Planes u;
  HIP_TRY(as_planes(block_hidden, cfg->dtype, p.u_in, u, st));
  return run_mamba_core(*cfg, *w, u, p, nullptr, 0, out, S_final, st);
}

HSPEC_API size_t hspec_target_kv_block_attn_workspace(const hspec_attn_cfg* cfg, int max_ctx_len) {
  if (!cfg) return 0;
  Arena ar;
  status_word(ar);
  AttnPlan p;
  plan_attn(ar, *cfg, max_ctx_len < 0 ? 0 : max_ctx_len, false, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_target_kv_block_attn(const hspec_attn_cfg* cfg, const hspec_attn_w* w, const void* x,
                                                  const void* k_cache, const void* v_cache,
                                                  const int32_t* page_table, const int32_t* ctx_lens,
                                                  int max_ctx_len, float* out, void* workspace, size_t ws_bytes,
                                                  void* stream) {
  clear_err();
  if (hspec_status s = check_attn_cfg(cfg, max_ctx_len)) return s;
  if (hspec_status s = check_attn_w(cfg, w)) return s;
  if (!x || !k_cache || !v_cache || !page_table || !ctx_lens || !out)
    return fail(HSPEC_ERR_NULL, "an input or output pointer is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_target_kv_block_attn_workspace(cfg, max_ctx_len)))
    return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  AttnPlan p;
  plan_attn(ar, *cfg, max_ctx_len, false, p);
  // no kernel before the work list sets a status bit: the work list clears the status words
  Planes xn;
  HIP_TRY(as_planes(x, cfg->dtype, p.x_in, xn, st));
  return run_attn_core(*cfg, *w, xn, k_cache, v_cache, page_table, ctx_lens, max_ctx_len, p, nullptr, 0, out, status,
                       hspec::kStatusClear, st);
}

HSPEC_API size_t hspec_draft_step_workspace(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg,
                                            int max_ctx_len) {
  if (!mcfg || !acfg) return 0;
  Arena ar;
  status_word(ar);
  DraftPlan p;
  plan_draft(ar, *mcfg, *acfg, max_ctx_len < 0 ? 0 : max_ctx_len, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_draft_step(const hspec_mamba_cfg* mcfg, const hspec_mamba_w* mw, const float* norm1_w,
                                        const hspec_attn_cfg* acfg, const hspec_attn_w* aw, const float* norm2_w,
                                        const void* h_last, const void* block_emb, const void* k_cache,
                                        const void* v_cache, const int32_t* page_table, const int32_t* ctx_lens,
                                        int max_ctx_len, float* out, void* workspace, size_t ws_bytes, void* stream) {
  clear_err();
  if (hspec_status s = check_mamba(mcfg, mw, true)) return s;
  if (hspec_status s = check_attn_cfg(acfg, max_ctx_len)) return s;
  if (hspec_status s = check_attn_w(acfg, aw)) return s;
  if (mcfg->B != acfg->B || mcfg->k != acfg->k || mcfg->d_model != acfg->d_model)
    return fail(HSPEC_ERR_SHAPE, "mamba and attention configs disagree on B, k or d_model");
  if (mcfg->dtype != acfg->dtype) return fail(HSPEC_ERR_DTYPE, "mamba and attention dtypes differ");
  if (!norm1_w || !norm2_w || !h_last || !block_emb || !k_cache || !v_cache || !page_table || !ctx_lens || !out)
    return fail(HSPEC_ERR_NULL, "an input or output pointer is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_draft_step_workspace(mcfg, acfg, max_ctx_len))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  DraftPlan p;
  plan_draft(ar, *mcfg, *acfg, max_ctx_len, p);
  const int M = mcfg->B * mcfg->k;
  const bool f32 = is_f32(mcfg->dtype);
  // no kernel before the attention's work list sets a status bit: the work list clears them
  if (hspec_status s = run_state(*mcfg, *mw, h_last, p.m.st, nullptr, st)) return s;
  HIP_TRY(hspec::launch_rmsnorm_planes(block_emb, !f32, norm1_w, M, mcfg->d_model, mcfg->eps, p.m.u_hi, p.m.u_lo, st));
  Planes u{p.m.u_hi, p.m.u_lo};
  if (hspec_status s = run_mamba_core(*mcfg, *mw, u, p.m, block_emb, !f32, p.x1, nullptr, st)) return s;
  HIP_TRY(hspec::launch_rmsnorm_planes(p.x1, 0, norm2_w, M, acfg->d_model, acfg->eps, p.at.xn_hi, p.at.xn_lo, st));
  Planes xn{p.at.xn_hi, p.at.xn_lo};
  return run_attn_core(*acfg, *aw, xn, k_cache, v_cache, page_table, ctx_lens, max_ctx_len, p.at, p.x1, 0, out, status,
                       hspec::kStatusClear, st);
}

HSPEC_API size_t hspec_ssd_scan_workspace(int B, int T, int H, int P, int N, int G, hspec_dtype dtype) {
  Arena ar;
  status_word(ar);
  if (dtype == HSPEC_F32 && B > 0 && T > 0) {
    reserve_split(ar, dtype, (size_t)B * T * H * P);
    reserve_split(ar, dtype, (size_t)B * T * G * N);
    reserve_split(ar, dtype, (size_t)B * T * G * N);
    reserve_split(ar, dtype, (size_t)B * H * P * N);
  }
  return ar.size();
}

HSPEC_API hspec_status hspec_ssd_scan(int B, int T, int H, int P, int N, int G, int chunk, hspec_dtype dtype,
                                      const void* x, const float* dt, const float* A, const void* Bm, const void* Cm,
                                      const float* Dskip, const void* S0, float* y, float* S_final, void* workspace,
                                      size_t ws_bytes, void* stream) {
  clear_err();
  if (!dtype_ok(dtype)) return fail(HSPEC_ERR_DTYPE, "unknown dtype %d", (int)dtype);
  if (B <= 0 || T <= 0 || H <= 0 || P <= 0 || N <= 0 || G <= 0 || chunk <= 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive scan dimension");
  if (H % G) return fail(HSPEC_ERR_SHAPE, "H %% G != 0");
  if (P != 64) return fail(HSPEC_ERR_UNSUPPORTED, "P must be 64, got %d", P);
  if (N != 16 && N != 32 && N != 64 && N != 128) return fail(HSPEC_ERR_UNSUPPORTED, "N must be 16/32/64/128");
  if (chunk > 16) return fail(HSPEC_ERR_UNSUPPORTED, "chunk must be <= 16");
  if (!x || !dt || !A || !Bm || !Cm || !Dskip || !y) return fail(HSPEC_ERR_NULL, "a scan pointer is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_ssd_scan_workspace(B, T, H, P, N, G, dtype))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  SplitSlot sx, sb, sc, ss;
  if (dtype == HSPEC_F32) {
    sx = reserve_split(ar, dtype, (size_t)B * T * H * P);
    sb = reserve_split(ar, dtype, (size_t)B * T * G * N);
    sc = reserve_split(ar, dtype, (size_t)B * T * G * N);
    ss = reserve_split(ar, dtype, (size_t)B * H * P * N);
  }
  HIP_TRY(hspec::launch_zero_words(status, hspec::kStatusClear, st));
  Planes px, pb, pc, ps;
  HIP_TRY(as_planes(x, dtype, sx, px, st));
  HIP_TRY(as_planes(Bm, dtype, sb, pb, st));
  HIP_TRY(as_planes(Cm, dtype, sc, pc, st));
  if (S0) HIP_TRY(as_planes(S0, dtype, ss, ps, st));
  hspec::ScanArgs a;
  a.x_hi = px.hi; a.x_lo = px.lo; a.dt = dt; a.A = A; a.A_is_log = 0;
  a.B_hi = pb.hi; a.B_lo = pb.lo; a.C_hi = pc.hi; a.C_lo = pc.lo; a.Dskip = Dskip;
  a.S0_hi = S0 ? ps.hi : nullptr; a.S0_lo = S0 ? ps.lo : nullptr;
  a.y = y; a.S_final = S_final;
  a.B = B; a.T = T; a.H = H; a.P = P; a.N = N; a.G = G; a.chunk = chunk;
  a.x_ld = H * P; a.bc_ld = G * N; a.dt_ld = H;
  HIP_TRY(hspec::launch_ssd_scan(a, st));
  return HSPEC_OK;
}

HSPEC_API size_t hspec_paged_attn_workspace(const hspec_attn_cfg* cfg, int max_ctx_len) {
  if (!cfg) return 0;
  Arena ar;
  status_word(ar);
  AttnPlan p;
  const size_t M = (size_t)cfg->B * cfg->k;
  p.qin = reserve_split(ar, cfg->dtype, M * cfg->Hq * cfg->D);
  p.kbin = reserve_split(ar, cfg->dtype, M * cfg->Hkv * cfg->D);
  p.vbin = reserve_split(ar, cfg->dtype, M * cfg->Hkv * cfg->D);
  plan_sweep(ar, *cfg, max_ctx_len < 0 ? 0 : max_ctx_len, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_paged_attn_phase(const hspec_attn_cfg* cfg, const void* q, const void* k_blk,
                                              const void* v_blk, const void* k_cache, const void* v_cache,
                                              const int32_t* page_table, const int32_t* ctx_lens, int max_ctx_len,
                                              float* o, void* workspace, size_t ws_bytes, unsigned phases,
                                              void* stream) {
  clear_err();
  if (hspec_status s = check_attn_cfg(cfg, max_ctx_len)) return s;
  if (!q || !k_blk || !v_blk || !k_cache || !v_cache || !page_table || !ctx_lens || !o)
    return fail(HSPEC_ERR_NULL, "an input or output pointer is NULL");
  if (phases & ~(unsigned)(HSPEC_PHASE_WORKLIST | HSPEC_PHASE_SWEEP | HSPEC_PHASE_REDUCE))
    return fail(HSPEC_ERR_UNSUPPORTED, "unknown phase bits 0x%x", phases);
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_paged_attn_workspace(cfg, max_ctx_len))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  AttnPlan p;
  const size_t M = (size_t)cfg->B * cfg->k;
  p.qin = reserve_split(ar, cfg->dtype, M * cfg->Hq * cfg->D);
  p.kbin = reserve_split(ar, cfg->dtype, M * cfg->Hkv * cfg->D);
  p.vbin = reserve_split(ar, cfg->dtype, M * cfg->Hkv * cfg->D);
  plan_sweep(ar, *cfg, max_ctx_len, p);
  // the sweep's work list is the call's first kernel and clears the status words
  if (phases & HSPEC_PHASE_WORKLIST)
    HIP_TRY(hspec::launch_attention_plan(sweep_args(*cfg, p, page_table, ctx_lens, max_ctx_len, status),
                                         hspec::kStatusClear, st));
  if (!(phases & (HSPEC_PHASE_SWEEP | HSPEC_PHASE_REDUCE))) return HSPEC_OK;
  Planes pq, pk, pv, kc, vc;
  if (phases & HSPEC_PHASE_SWEEP) {
    HIP_TRY(as_planes(q, cfg->dtype, p.qin, pq, st));
    HIP_TRY(as_planes(k_blk, cfg->dtype, p.kbin, pk, st));
    HIP_TRY(as_planes(v_blk, cfg->dtype, p.vbin, pv, st));
    HIP_TRY(as_planes(k_cache, cfg->dtype, p.kc, kc, st));
    HIP_TRY(as_planes(v_cache, cfg->dtype, p.vc, vc, st));
  } else {
    // the reduction alone still reads the block q, k and v: the caller's bf16 tensors, or the
    // planes the sweep phase of this attention wrote into the workspace (fp32 storage)
    pq = planes_in_place(q, cfg->dtype, p.qin);
    pk = planes_in_place(k_blk, cfg->dtype, p.kbin);
    pv = planes_in_place(v_blk, cfg->dtype, p.vbin);
  }
  hspec::AttnArgs a = sweep_args(*cfg, p, page_table, ctx_lens, max_ctx_len, status);
  a.q_hi = pq.hi; a.q_lo = pq.lo; a.kb_hi = pk.hi; a.kb_lo = pk.lo; a.vb_hi = pv.hi; a.vb_lo = pv.lo;
  a.kc_hi = kc.hi; a.kc_lo = kc.lo; a.vc_hi = vc.hi; a.vc_lo = vc.lo;
  a.o_f32 = o;
  const unsigned parts = ((phases & HSPEC_PHASE_SWEEP) ? hspec::ATTN_SWEEP : 0u) |
                         ((phases & HSPEC_PHASE_REDUCE) ? hspec::ATTN_REDUCE : 0u);
  HIP_TRY(hspec::launch_attention(a, st, parts));
  return HSPEC_OK;
}

HSPEC_API hspec_status hspec_paged_attn(const hspec_attn_cfg* cfg, const void* q, const void* k_blk,
                                        const void* v_blk, const void* k_cache, const void* v_cache,
                                        const int32_t* page_table, const int32_t* ctx_lens, int max_ctx_len, float* o,
                                        void* workspace, size_t ws_bytes, void* stream) {
  return hspec_paged_attn_phase(cfg, q, k_blk, v_blk, k_cache, v_cache, page_table, ctx_lens, max_ctx_len, o,
                                workspace, ws_bytes, HSPEC_PHASE_WORKLIST | HSPEC_PHASE_SWEEP | HSPEC_PHASE_REDUCE,
                                stream);
}

HSPEC_API hspec_status hspec_gather_slots(int B, int max_pages, int page_size, int num_pages,
                                          const int32_t* page_table, const int32_t* ctx_lens, int max_ctx_len,
                                          int32_t* slots, int32_t* status, void* stream) {
  clear_err();
  if (B <= 0 || max_pages <= 0 || page_size <= 0 || num_pages <= 0 || max_ctx_len < 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive gather dimension");
  if (!page_table || !ctx_lens || (!slots && max_ctx_len > 0)) return fail(HSPEC_ERR_NULL, "a gather pointer is NULL");
  if (page_size < 16 || (page_size & (page_size - 1)))
    return fail(HSPEC_ERR_UNSUPPORTED, "page_size must be a power of two >= 16, got %d", page_size);
  HIP_TRY(hspec::launch_gather_slots(B, max_pages, page_size, num_pages, page_table, ctx_lens, max_ctx_len, slots,
                                     status, (hipStream_t)stream));
  return HSPEC_OK;
}

HSPEC_API size_t hspec_linear_workspace(hspec_dtype dtype, int M, int N, int K) {
  Arena ar;
  status_word(ar);
  if (M > 0 && N > 0 && K > 0) {
    reserve_split(ar, dtype, (size_t)M * K);
    reserve_split(ar, dtype, (size_t)N * K);
    reserve_gemm(ar, dtype, {{M, N, K}});
  }
  return ar.size();
}

HSPEC_API hspec_status hspec_linear(hspec_dtype dtype, int M, int N, int K, const void* A, const void* W,
                                    const float* R, float* C, void* workspace, size_t ws_bytes, void* stream) {
  clear_err();
  if (!dtype_ok(dtype)) return fail(HSPEC_ERR_DTYPE, "unknown dtype %d", (int)dtype);
  if (M <= 0 || N <= 0 || K <= 0) return fail(HSPEC_ERR_SHAPE, "non-positive GEMM dimension");
  if (K % 8) return fail(HSPEC_ERR_UNSUPPORTED, "K must be a multiple of 8");
  if (!A || !W || !C) return fail(HSPEC_ERR_NULL, "A, W or C is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_linear_workspace(dtype, M, N, K))) return s;
  hipStream_t st = (hipStream_t)stream;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  SplitSlot sa = reserve_split(ar, dtype, (size_t)M * K), sw = reserve_split(ar, dtype, (size_t)N * K);
  const GemmScratch gs = reserve_gemm(ar, dtype, {{M, N, K}});
  HIP_TRY(hspec::launch_zero_words(status, hspec::kStatusClear, st));
  Planes pa, pw;
  HIP_TRY(as_planes(A, dtype, sa, pa, st));
  HIP_TRY(as_planes(W, dtype, sw, pw, st));
  hspec::GemmArgs g;
  g.A_hi = pa.hi; g.A_lo = pa.lo; g.lda = K;
  g.W_hi = pw.hi; g.W_lo = pw.lo; g.ldw = K;
  g.M = M; g.N = N; g.K = K;
  g.C = C; g.ldc = N; g.R = R; g.ldr = N; g.r_bf16 = 0;
  use_scratch(g, gs);
  HIP_TRY(hspec::launch_gemm(g, st));
  return HSPEC_OK;
}

// ---------------------------------------------------------------- whole drafter forward

struct ForwardPlan {
  MambaPlan m;                              // with the state plan; its u planes also feed the MLP
  AttnPlan at;
  float *xa = nullptr, *xb = nullptr;       // residual stream, alternating
  SplitSlot wg, wu, wd;
  float* gu = nullptr;                      // [M, 2 ff]: gate | up
  bf16 *h_hi = nullptr, *h_lo = nullptr;    // [M, ff]
  GemmScratch gs;
};

void plan_forward(Arena& ar, const hspec_mamba_cfg& mc, const hspec_attn_cfg& ac, int ff, int max_ctx_len,
                  ForwardPlan& p) {
  plan_mamba(ar, mc, true, p.m);
  plan_attn(ar, ac, max_ctx_len, true, p.at);
  const size_t M = (size_t)mc.B * mc.k;
  p.xa = ar.take<float>(M * mc.d_model);
  p.xb = ar.take<float>(M * mc.d_model);
  p.wg = reserve_split(ar, mc.dtype, (size_t)ff * mc.d_model);
  p.wu = reserve_split(ar, mc.dtype, (size_t)ff * mc.d_model);
  p.wd = reserve_split(ar, mc.dtype, (size_t)mc.d_model * ff);
  p.gu = ar.take<float>(M * 2 * ff);
  p.h_hi = ar.take<bf16>(M * ff);
  p.h_lo = ar.take<bf16>(M * ff);
  p.gs = reserve_gemm(ar, mc.dtype, {{(int)M, 2 * ff, mc.d_model}, {(int)M, ff, mc.d_model}, {(int)M, mc.d_model, ff}});
}

// x_out = x + W_down (SiLU(W_gate u) * (W_up u)), u already normalised (planes).
hspec_status run_mlp(const hspec_mamba_cfg& c, const hspec_layer_w& L, int ff, Planes u, const ForwardPlan& p,
                     const void* x, int x_bf16, float* x_out, hipStream_t st) {
  const int M = c.B * c.k;
  Planes wg, wu, wd;
  HIP_TRY(as_planes(L.W_gate, c.dtype, p.wg, wg, st));
  HIP_TRY(as_planes(L.W_up, c.dtype, p.wu, wu, st));
  HIP_TRY(as_planes(L.W_down, c.dtype, p.wd, wd, st));
  if (!wg.lo) {
    // one product over the two row segments [W_gate; W_up]
    hspec::GemmArgs g;
    g.A_hi = u.hi; g.A_lo = u.lo; g.lda = c.d_model;
    g.W_hi = wg.hi; g.W2 = wu.hi; g.N1 = ff; g.N2 = ff; g.ldw = c.d_model;
    g.M = M; g.N = 2 * ff; g.K = c.d_model;
    g.C = p.gu; g.ldc = 2 * ff;
    use_scratch(g, p.gs);
    HIP_TRY(hspec::launch_gemm(g, st));
  } else {
    const Planes* w2[2] = {&wg, &wu};
    for (int i = 0; i < 2; ++i) {
      hspec::GemmArgs g;
      g.A_hi = u.hi; g.A_lo = u.lo; g.lda = c.d_model;
      g.W_hi = w2[i]->hi; g.W_lo = w2[i]->lo; g.ldw = c.d_model;
      g.M = M; g.N = ff; g.K = c.d_model;
      g.C = p.gu + (size_t)i * ff; g.ldc = 2 * ff;
      use_scratch(g, p.gs);
      HIP_TRY(hspec::launch_gemm(g, st));
    }
  }
  HIP_TRY(hspec::launch_silu_mul(p.gu, M, ff, p.h_hi, p.h_lo, st));
  hspec::GemmArgs g;
  g.A_hi = p.h_hi; g.A_lo = p.h_lo; g.lda = ff;
  g.W_hi = wd.hi; g.W_lo = wd.lo; g.ldw = ff;
  g.M = M; g.N = c.d_model; g.K = ff;
  g.C = x_out; g.ldc = c.d_model;
  g.R = x; g.ldr = c.d_model; g.r_bf16 = x_bf16;
  use_scratch(g, p.gs);
  HIP_TRY(hspec::launch_gemm(g, st));
  return HSPEC_OK;
}

HSPEC_API size_t hspec_drafter_forward_workspace(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg, int ff,
                                                 int max_ctx_len) {
  if (!mcfg || !acfg || ff <= 0) return 0;
  hspec_mamba_cfg mc = *mcfg;
  mc.flags |= HSPEC_MAMBA_PRECISE_IO;
  hspec_attn_cfg ac = *acfg;
  ac.flags |= HSPEC_ATTN_PRECISE_IO;
  Arena ar;
  status_word(ar);
  ForwardPlan p;
  plan_forward(ar, mc, ac, ff, max_ctx_len < 0 ? 0 : max_ctx_len, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_drafter_forward(const hspec_mamba_cfg* mcfg, const hspec_attn_cfg* acfg, int ff,
                                             int n_layers, const void* W_r, const void* W_dS,
                                             const hspec_layer_w* layers, const void* h_last, const void* block_emb,
                                             const int32_t* page_table, const int32_t* ctx_lens, int max_ctx_len,
                                             float* out, void* workspace, size_t ws_bytes, void* stream) {
  clear_err();
  if (!mcfg || !acfg) return fail(HSPEC_ERR_NULL, "mamba or attention config is NULL");
  if (n_layers < 1) return fail(HSPEC_ERR_SHAPE, "n_layers must be >= 1");
  if (!layers) return fail(HSPEC_ERR_NULL, "layers is NULL");
  if (ff <= 0) return fail(HSPEC_ERR_SHAPE, "ff must be positive");
  if (ff % 8) return fail(HSPEC_ERR_UNSUPPORTED, "ff must be a multiple of 8");
  bool any_attn = false, any_mamba = false;
  for (int l = 0; l < n_layers; ++l) {
    const hspec_layer_w& L = layers[l];
    if (L.mamba) {
      any_mamba = true;
      hspec_mamba_w mw = *L.mamba;
      mw.W_r = W_r;
      mw.W_dS = W_dS;
      if (hspec_status s = check_mamba(mcfg, &mw, true)) return s;
      if (!L.norm1_w) return fail(HSPEC_ERR_NULL, "layer %d: norm1_w is NULL", l);
    }
    if (!L.norm3_w || !L.W_gate || !L.W_up || !L.W_down)
      return fail(HSPEC_ERR_NULL, "layer %d: a norm or MLP weight is NULL", l);
    if (L.attn) {
      any_attn = true;
      if (hspec_status s = check_attn_w(acfg, L.attn)) return s;
      if (!L.norm2_w || !L.k_cache || !L.v_cache) return fail(HSPEC_ERR_NULL, "layer %d: attention input is NULL", l);
    }
  }
  if (hspec_status s = check_attn_cfg(acfg, max_ctx_len)) return s;
  if (mcfg->B != acfg->B || mcfg->k != acfg->k || mcfg->d_model != acfg->d_model)
    return fail(HSPEC_ERR_SHAPE, "mamba and attention configs disagree on B, k or d_model");
  if (mcfg->dtype != acfg->dtype) return fail(HSPEC_ERR_DTYPE, "mamba and attention dtypes differ");
  if (!any_mamba && (mcfg->B <= 0 || mcfg->k <= 0 || mcfg->d_model <= 0 || mcfg->d_model % 8 || !dtype_ok(mcfg->dtype)))
    return fail(HSPEC_ERR_SHAPE, "bad B, k, d_model or dtype");
  if (!block_emb || !out || (any_mamba && !h_last) || (any_attn && (!page_table || !ctx_lens)))
    return fail(HSPEC_ERR_NULL, "an input or output pointer is NULL");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_drafter_forward_workspace(mcfg, acfg, ff, max_ctx_len)))
    return s;
  hipStream_t st = (hipStream_t)stream;
  // the layers' errors add up over the stack: activations enter every projection as hi/lo planes
  hspec_mamba_cfg mc = *mcfg;
  mc.flags |= HSPEC_MAMBA_PRECISE_IO;
  hspec_attn_cfg ac = *acfg;
  ac.flags |= HSPEC_ATTN_PRECISE_IO;
  Arena ar{(char*)workspace};
  int* status = status_word(ar);
  ForwardPlan p;
  plan_forward(ar, mc, ac, ff, max_ctx_len, p);
  const int M = mc.B * mc.k;
  const bool f32 = is_f32(mc.dtype);
  HIP_TRY(hspec::launch_zero_words(status, hspec::kStatusClear, st));
  if (any_mamba) {
    hspec_mamba_w sw{};
    sw.W_r = W_r;
    sw.W_dS = W_dS;
    if (hspec_status s = run_state(mc, sw, h_last, p.m.st, nullptr, st)) return s;
  }

  // the residual stream: block_emb (storage dtype), then fp32 buffers; the last sublayer
  // writes straight into out
  int total = 0;
  for (int l = 0; l < n_layers; ++l) total += 1 + (layers[l].mamba ? 1 : 0) + (layers[l].attn ? 1 : 0);
  int done = 0;
  const void* x = block_emb;
  int x_bf16 = !f32;
  auto dst = [&]() -> float* { return ++done == total ? out : (x == p.xa ? p.xb : p.xa); };
  Planes u{p.m.u_hi, p.m.u_lo};
  for (int l = 0; l < n_layers; ++l) {
    const hspec_layer_w& L = layers[l];
    float* y = nullptr;
    if (L.mamba) {
      HIP_TRY(hspec::launch_rmsnorm_planes(x, x_bf16, L.norm1_w, M, mc.d_model, mc.eps, p.m.u_hi, p.m.u_lo, st));
      y = dst();
      if (hspec_status s = run_mamba_core(mc, *L.mamba, u, p.m, x, x_bf16, y, nullptr, st)) return s;
      x = y;
      x_bf16 = 0;
    }
    if (L.attn) {
      HIP_TRY(hspec::launch_rmsnorm_planes(x, x_bf16, L.norm2_w, M, ac.d_model, ac.eps, p.at.xn_hi, p.at.xn_lo, st));
      Planes xn{p.at.xn_hi, p.at.xn_lo};
      y = dst();
      if (hspec_status s = run_attn_core(ac, *L.attn, xn, L.k_cache, L.v_cache, page_table, ctx_lens, max_ctx_len,
                                         p.at, x, x_bf16, y, status, 0, st))   // work list, fresh queue
        return s;
      x = y;
      x_bf16 = 0;
    }
    HIP_TRY(hspec::launch_rmsnorm_planes(x, x_bf16, L.norm3_w, M, mc.d_model, mc.eps, p.m.u_hi, p.m.u_lo, st));
    y = dst();
    if (hspec_status s = run_mlp(mc, L, ff, u, p, x, x_bf16, y, st)) return s;
    x = y;
    x_bf16 = 0;
  }
  return HSPEC_OK;
}

// ------------------------------------------------ drafter-side KV injection (comparison)

struct InjectPlan {
  int* status = nullptr;
  SplitSlot h, wfc, wk, wv;
  float* f = nullptr;                        // fused [M, d_model]
  bf16 *f_hi = nullptr, *f_lo = nullptr;
  float* kv = nullptr;                       // [M, 2 Hkv D]: k | v of one layer
  bf16 *k_hi = nullptr, *k_lo = nullptr, *v_hi = nullptr, *v_lo = nullptr;
  GemmScratch gs;
};

void plan_inject(Arena& ar, const hspec_attn_cfg& c, int d_h, InjectPlan& p) {
  p.status = status_word(ar);
  const size_t M = (size_t)c.B * c.k, kvw = (size_t)c.Hkv * c.D;
  p.h = reserve_split(ar, c.dtype, M * d_h);
  p.wfc = reserve_split(ar, c.dtype, (size_t)c.d_model * d_h);
  p.wk = reserve_split(ar, c.dtype, kvw * c.d_model);
  p.wv = reserve_split(ar, c.dtype, kvw * c.d_model);
  p.f = ar.take<float>(M * c.d_model);
  p.f_hi = ar.take<bf16>(M * c.d_model);
  p.f_lo = ar.take<bf16>(M * c.d_model);
  p.kv = ar.take<float>(M * 2 * kvw);
  p.k_hi = ar.take<bf16>(M * kvw);
  p.k_lo = ar.take<bf16>(M * kvw);
  p.v_hi = ar.take<bf16>(M * kvw);
  p.v_lo = ar.take<bf16>(M * kvw);
  p.gs = reserve_gemm(ar, c.dtype, {{(int)M, c.d_model, d_h}, {(int)M, 2 * (int)kvw, c.d_model}, {(int)M, (int)kvw, c.d_model}});
}

HSPEC_API size_t hspec_kv_inject_workspace(const hspec_attn_cfg* cfg, int d_h) {
  if (!cfg || d_h <= 0 || cfg->B <= 0 || cfg->k <= 0) return 0;
  Arena ar;
  InjectPlan p;
  plan_inject(ar, *cfg, d_h, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_kv_inject(const hspec_attn_cfg* cfg, int d_h, int n_layers, const void* h_new,
                                       const void* W_fc, const void* const* W_k, const void* const* W_v,
                                       const float* const* k_norm_w, void* const* k_cache, void* const* v_cache,
                                       const int32_t* page_table, const int32_t* ctx_lens, void* workspace,
                                       size_t ws_bytes, void* stream) {
  clear_err();
  if (hspec_status s = check_attn_cfg(cfg, 0)) return s;
  if (cfg->kv_heads || (cfg->Hkv_cache != 0 && cfg->Hkv_cache != cfg->Hkv))
    return fail(HSPEC_ERR_UNSUPPORTED, "KV injection writes the drafter's own caches: no KV-head subset");
  if (d_h <= 0 || n_layers < 1) return fail(HSPEC_ERR_SHAPE, "d_h and n_layers must be positive");
  if (d_h % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_h must be a multiple of 8");
  if (cfg->d_model <= 0 || cfg->d_model % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_model must be a positive multiple of 8");
  if (!h_new || !W_fc || !W_k || !W_v || !k_norm_w || !k_cache || !v_cache || !page_table || !ctx_lens)
    return fail(HSPEC_ERR_NULL, "an input or output pointer is NULL");
  for (int l = 0; l < n_layers; ++l)
    if (!W_k[l] || !W_v[l] || !k_norm_w[l] || !k_cache[l] || !v_cache[l])
      return fail(HSPEC_ERR_NULL, "layer %d: a weight or cache pointer is NULL", l);
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_kv_inject_workspace(cfg, d_h))) return s;
  hipStream_t st = (hipStream_t)stream;
  const hspec_attn_cfg& c = *cfg;
  Arena ar{(char*)workspace};
  InjectPlan p;
  plan_inject(ar, c, d_h, p);
  HIP_TRY(hspec::launch_zero_words(p.status, hspec::kStatusClear, st));
  const int M = c.B * c.k, kvw = c.Hkv * c.D;
  Planes h, wfc;
  HIP_TRY(as_planes(h_new, c.dtype, p.h, h, st));
  HIP_TRY(as_planes(W_fc, c.dtype, p.wfc, wfc, st));
  hspec::GemmArgs g;
  g.A_hi = h.hi; g.A_lo = h.lo; g.lda = d_h;
  g.W_hi = wfc.hi; g.W_lo = wfc.lo; g.ldw = d_h;
  g.M = M; g.N = c.d_model; g.K = d_h;
  g.C = p.f; g.ldc = c.d_model;
  use_scratch(g, p.gs);
  HIP_TRY(hspec::launch_gemm(g, st));
  HIP_TRY(hspec::launch_split_planes(p.f, (size_t)M * c.d_model, p.f_hi, p.f_lo, st));
  for (int l = 0; l < n_layers; ++l) {
    Planes wk, wv;
    HIP_TRY(as_planes(W_k[l], c.dtype, p.wk, wk, st));
    HIP_TRY(as_planes(W_v[l], c.dtype, p.wv, wv, st));
    if (!wk.lo) {   // one product over the two row segments [W_k; W_v]
      hspec::GemmArgs gk;
      gk.A_hi = p.f_hi; gk.A_lo = p.f_lo; gk.lda = c.d_model;
      gk.W_hi = wk.hi; gk.W2 = wv.hi; gk.N1 = kvw; gk.N2 = kvw; gk.ldw = c.d_model;
      gk.M = M; gk.N = 2 * kvw; gk.K = c.d_model;
      gk.C = p.kv; gk.ldc = 2 * kvw;
      use_scratch(gk, p.gs);
      HIP_TRY(hspec::launch_gemm(gk, st));
    } else {
      const Planes* w2[2] = {&wk, &wv};
      for (int i = 0; i < 2; ++i) {
        hspec::GemmArgs gk;
        gk.A_hi = p.f_hi; gk.A_lo = p.f_lo; gk.lda = c.d_model;
        gk.W_hi = w2[i]->hi; gk.W_lo = w2[i]->lo; gk.ldw = c.d_model;
        gk.M = M; gk.N = kvw; gk.K = c.d_model;
        gk.C = p.kv + (size_t)i * kvw; gk.ldc = 2 * kvw;
        use_scratch(gk, p.gs);
        HIP_TRY(hspec::launch_gemm(gk, st));
      }
    }
    // k: per-head RMSNorm + RoPE at ctx_len + i (no query heads); v: copied
    HIP_TRY(hspec::launch_qk_norm_rope(p.kv, nullptr, k_norm_w[l], ctx_lens, c.B, c.k, 0, c.Hkv, c.D, c.eps,
                                       c.rope_theta, nullptr, nullptr, p.k_hi, p.k_lo, p.v_hi, p.v_lo, st));
    HIP_TRY(hspec::launch_kv_append(p.k_hi, p.k_lo, p.v_hi, p.v_lo, c.B, c.k, c.Hkv, c.D, page_table, c.max_pages,
                                    c.num_pages, c.page_size, ctx_lens, k_cache[l], v_cache[l], !is_f32(c.dtype),
                                    p.status, st));
  }
  return HSPEC_OK;
}

// ------------------------------------------------------------------------- draft head

hspec_status check_head(const hspec_head_cfg* c) {
  if (!c) return fail(HSPEC_ERR_NULL, "head config is NULL");
  if (c->B <= 0 || c->k <= 0 || c->d_model <= 0 || c->vocab <= 0 || c->rank <= 0)
    return fail(HSPEC_ERR_SHAPE, "non-positive head dimension");
  if (c->d_model % 8) return fail(HSPEC_ERR_UNSUPPORTED, "d_model must be a multiple of 8");
  if (c->rank % 32) return fail(HSPEC_ERR_UNSUPPORTED, "the Markov rank must be a multiple of 32");
  if ((long long)c->B * c->k > (1LL << 30) || (long long)c->vocab * c->rank > (1LL << 40))
    return fail(HSPEC_ERR_UNSUPPORTED, "head too large");
  return HSPEC_OK;
}

struct HeadPlan {
  int* status = nullptr;
  bf16* hn = nullptr;
  float* base = nullptr;
  unsigned long long* keys = nullptr;
  GemmScratch gs;
};

void plan_head(Arena& ar, const hspec_head_cfg& c, HeadPlan& p) {
  p.status = status_word(ar);
  const size_t M = (size_t)c.B * c.k;
  p.hn = ar.take<bf16>(M * c.d_model);
  p.base = ar.take<float>(M * c.vocab);
  p.keys = ar.take<unsigned long long>(M);
  p.gs = reserve_gemm(ar, HSPEC_BF16, {{(int)M, c.vocab, c.d_model}});
}

HSPEC_API size_t hspec_draft_head_workspace(const hspec_head_cfg* cfg) {
  if (!cfg || cfg->B <= 0 || cfg->k <= 0 || cfg->d_model <= 0 || cfg->vocab <= 0) return 0;
  Arena ar;
  HeadPlan p;
  plan_head(ar, *cfg, p);
  return ar.size();
}

HSPEC_API hspec_status hspec_draft_head(const hspec_head_cfg* cfg, const hspec_head_w* w, const float* hidden,
                                        const int32_t* prev_tok, const float* gumbel, const int32_t* forced,
                                        int32_t* tokens, float* logits, void* workspace, size_t ws_bytes,
                                        void* stream) {
  clear_err();
  if (hspec_status s = check_head(cfg)) return s;
  if (!w || !w->norm_f_w || !w->W_lm || !w->E_M || !w->U_M) return fail(HSPEC_ERR_NULL, "head weight is NULL");
  if (!hidden || !prev_tok || !tokens) return fail(HSPEC_ERR_NULL, "hidden, prev_tok or tokens is NULL");
  if (gumbel && !(cfg->temperature > 0.f)) return fail(HSPEC_ERR_SHAPE, "sampling needs temperature > 0");
  if (hspec_status s = check_ws(workspace, ws_bytes, hspec_draft_head_workspace(cfg))) return s;
  hipStream_t st = (hipStream_t)stream;
  const hspec_head_cfg& c = *cfg;
  Arena ar{(char*)workspace};
  HeadPlan p;
  plan_head(ar, c, p);
  hspec::HeadArgs h;
  h.B = c.B; h.k = c.k; h.V = c.vocab; h.R = c.rank;
  h.keys = p.keys; h.status = p.status;
  HIP_TRY(hspec::launch_head_clear(h, hspec::kStatusClear, st));
  const int M = c.B * c.k;
  HIP_TRY(hspec::launch_rmsnorm_planes(hidden, 0, w->norm_f_w, M, c.d_model, c.eps, p.hn, nullptr, st));
  // LM head over the pruned vocabulary; written straight into the caller's logits when given
  float* base = logits ? logits : p.base;
  hspec::GemmArgs g;
  g.A_hi = p.hn; g.lda = c.d_model;
  g.W_hi = static_cast<const bf16*>(w->W_lm); g.ldw = c.d_model;
  g.M = M; g.N = c.vocab; g.K = c.d_model;
  g.C = base; g.ldc = c.vocab;
  use_scratch(g, p.gs);
  HIP_TRY(hspec::launch_gemm(g, st));
  h.E = static_cast<const bf16*>(w->E_M); h.U = static_cast<const bf16*>(w->U_M);
  h.base = base; h.logits = logits; h.gumbel = gumbel;
  h.inv_temp = gumbel ? 1.f / c.temperature : 1.f;
  h.prev = prev_tok; h.forced = forced; h.tokens = tokens;
  HIP_TRY(hspec::launch_markov_head(h, st));
  return HSPEC_OK;
}

HSPEC_API size_t hspec_pack_w_ds_bytes(int d_S, int r) {
  if (d_S <= 0 || r <= 0 || d_S % 16 || r % 64) return 0;
  return (size_t)d_S * r * sizeof(bf16);
}

HSPEC_API hspec_status hspec_pack_w_ds(int d_S, int r, const void* W_dS, void* W_packed, void* stream) {
  clear_err();
  if (d_S <= 0 || r <= 0) return fail(HSPEC_ERR_SHAPE, "non-positive W_dS dimension");
  if (d_S % 16 || r % 64) return fail(HSPEC_ERR_UNSUPPORTED, "packing needs d_S %% 16 == 0 and r %% 64 == 0");
  if (!W_dS || !W_packed) return fail(HSPEC_ERR_NULL, "W_dS or W_packed is NULL");
  HIP_TRY(hspec::launch_pack_w(static_cast<const bf16*>(W_dS), d_S, r, static_cast<_Float16*>(W_packed),
                               (hipStream_t)stream));
  return HSPEC_OK;
}

HSPEC_API hspec_status hspec_read_status(const void* workspace, int32_t* status, void* stream) {
  clear_err();
  if (!workspace || !status) return fail(HSPEC_ERR_NULL, "workspace or status is NULL");
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(status, workspace, sizeof(int32_t), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  return HSPEC_OK;
}

HSPEC_API const char* hspec_status_string(hspec_status s) {
  switch (s) {
    case HSPEC_OK: return "ok";
    case HSPEC_ERR_NULL: return "null pointer";
    case HSPEC_ERR_SHAPE: return "bad shape";
    case HSPEC_ERR_DTYPE: return "bad dtype";
    case HSPEC_ERR_UNSUPPORTED: return "unsupported dimension";
    case HSPEC_ERR_WORKSPACE: return "workspace too small or misaligned";
    case HSPEC_ERR_LAUNCH: return "kernel launch failed";
  }
  return "unknown status";
}

HSPEC_API const char* hspec_last_error(void) { return g_err; }

namespace hspec {
hspec_status api_fail(hspec_status s, const char* msg) { return fail(s, "%s", msg); }
}  // namespace hspec
