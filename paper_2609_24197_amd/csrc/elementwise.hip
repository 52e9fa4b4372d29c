// Normalisation, convolution and rotary kernels of the drafting step, plus small helpers.
// Each writes its result as bf16 planes ready to be MFMA operands (hi, and lo = rounding
// residual where the next contraction needs fp32-level accuracy).
#include "common.h"
#include "kernels.h"
#include "worklist.h"

namespace hspec {

namespace {

__device__ __forceinline__ void put_planes(bf16* hi, bf16* lo, size_t i, float v) {
  const bf16 h = f2bf(v);
  hi[i] = h;
  if (lo) lo[i] = f2bf(v - bf2f(h));
}

__device__ __forceinline__ float silu(float v) { return v / (1.f + __expf(-v)); }
__device__ __forceinline__ float softplus(float v) {
  return fmaxf(v, 0.f) + log1pf(__expf(-fabsf(v)));
}

// Block-wide sum for 256 threads.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  __syncthreads();
  return t;
}

// 8 consecutive elements as fp32 (one 16-byte bf16 load or two 16-byte fp32 loads).
__device__ __forceinline__ void load8(const bf16* p, float (&v)[8]) {
  const bf16x8 x = ld8(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = bf2f(x[e]);
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = a[e];
    v[4 + e] = b[e];
  }
}
__device__ __forceinline__ void put8(bf16* hi, bf16* lo, size_t i, const float (&v)[8]) {
  bf16x8 h, l;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = f2bf(v[e]);
    l[e] = f2bf(v[e] - bf2f(h[e]));
  }
  *reinterpret_cast<bf16x8*>(hi + i) = h;
  if (lo) *reinterpret_cast<bf16x8*>(lo + i) = l;
}

// One workgroup per row, 8 elements per thread and step (n % 8 == 0).  NR > 0: the row fits in
// NR chunks of 8 per thread (n <= 2048 NR); every chunk is loaded before the sum of squares and
// kept in registers for the scaling pass (chunks past the row end load the row's first chunk and
// count as zero).  NR == 0: any n, the second pass re-reads the row from cache.
template <typename T, int NR>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const T* x, const float* w, int n, float eps,
                                                      bf16* hi, bf16* lo) {
  __shared__ float red[4];
  const size_t row = blockIdx.x;
  const T* xr = x + row * n;
  if constexpr (NR > 0) {
    float v[NR][8];
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NR; ++c) {
      const int i = (threadIdx.x + c * 256) * 8;
      load8(xr + (i < n ? i : 0), v[c]);
    }
#pragma unroll
    for (int c = 0; c < NR; ++c)
      if ((threadIdx.x + c * 256) * 8 < n)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[c][e] * v[c][e];
    ss = block_sum(ss, red);
    const float r = rsqrtf(ss / n + eps);
#pragma unroll
    for (int c = 0; c < NR; ++c) {
      const int i = (threadIdx.x + c * 256) * 8;
      if (i >= n) break;
      float g[8];
      load8(w + i, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = v[c][e] * r * g[e];
      put8(hi, lo, row * n + i, v[c]);
    }
    return;
  }
  float ss = 0.f;
  for (int i = threadIdx.x * 8; i < n; i += blockDim.x * 8) {
    float v[8];
    load8(xr + i, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  ss = block_sum(ss, red);
  const float r = rsqrtf(ss / n + eps);
  for (int i = threadIdx.x * 8; i < n; i += blockDim.x * 8) {
    float v[8], g[8];
    load8(xr + i, v);
    load8(w + i, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * g[e];
    put8(hi, lo, row * n + i, v);
  }
}

template <typename T>
__global__ void __launch_bounds__(256) conv_split_kernel(ConvArgs a) {
  const int di = a.H * a.P, gn = a.G * a.N, cdim = di + 2 * gn;
  const int dproj = 2 * di + 2 * gn + a.H;
  const int tok = blockIdx.y;                        // b*T + t
  const int t = tok % a.T;
  const T* cw = reinterpret_cast<const T*>(a.conv_w);
  const T* cb = reinterpret_cast<const T*>(a.conv_b);
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < cdim + a.H; c += gridDim.x * blockDim.x) {
    if (c < cdim) {
      float v = to_f32(cb[c]);
      for (int j = 0; j < a.K; ++j) {
        const int tau = t - (a.K - 1) + j;
        if (tau >= 0) v += to_f32(cw[(size_t)c * a.K + j]) * a.zxbcdt[(size_t)(tok - t + tau) * dproj + di + c];
      }
      v = silu(v);
      if (c < di) put_planes(a.x_hi, a.x_lo, (size_t)tok * di + c, v);
      else if (c < di + gn) put_planes(a.B_hi, a.B_lo, (size_t)tok * gn + (c - di), v);
      else put_planes(a.C_hi, a.C_lo, (size_t)tok * gn + (c - di - gn), v);
    } else {
      const int hh = c - cdim;
      a.dt[(size_t)tok * a.H + hh] = softplus(a.zxbcdt[(size_t)tok * dproj + 2 * di + 2 * gn + hh] + a.dt_bias[hh]);
    }
  }
}

// Causal conv with the paper's width of 4 taps: a thread owns 4 consecutive channels of
// CONV_TT consecutive tokens of one request and reads the CONV_TT + 3 inputs they need (tokens
// before the block's first are zero) straight from zx, all loads in flight together.  Weights of
// the 4 channels are 16 consecutive values, read as vectors.  Same alignment needs as the serial
// kernel below.
constexpr int CONV_TT = 4;

template <typename T>
__global__ void __launch_bounds__(256) conv4_tok_kernel(ConvArgs a) {
  const int di = a.H * a.P, gn = a.G * a.N, cdim = di + 2 * gn;
  const int dproj = 2 * di + 2 * gn + a.H;
  const int nq = (a.T + CONV_TT - 1) / CONV_TT;
  const int b = blockIdx.y / nq, t0 = (blockIdx.y % nq) * CONV_TT;
  const int c = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (c >= cdim + a.H) return;
  const float* zb = a.zxbcdt + (size_t)b * a.T * dproj;
  if (c >= cdim) {                                   // dt = softplus(dt_raw + dt_bias), 4 heads
    const int hh = c - cdim;
    f32x4 v[CONV_TT];
#pragma unroll
    for (int u = 0; u < CONV_TT; ++u)
      v[u] = t0 + u < a.T ? *reinterpret_cast<const f32x4*>(zb + (size_t)(t0 + u) * dproj + 2 * di + 2 * gn + hh)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < CONV_TT; ++u) {
      if (t0 + u >= a.T) break;
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = softplus(v[u][e] + a.dt_bias[hh + e]);
      *reinterpret_cast<f32x4*>(a.dt + ((size_t)b * a.T + t0 + u) * a.H + hh) = o;
    }
    return;
  }
  // in[j] is token t0 - 3 + j
  f32x4 in[CONV_TT + 3];
#pragma unroll
  for (int j = 0; j < CONV_TT + 3; ++j) {
    const int tau = t0 - 3 + j;
    in[j] = tau >= 0 && tau < a.T ? *reinterpret_cast<const f32x4*>(zb + (size_t)tau * dproj + di + c)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float w[16], bias[4];
  if constexpr (sizeof(T) == 2) {
    const bf16x8 w0 = ld8(reinterpret_cast<const bf16*>(a.conv_w) + (size_t)c * 4);
    const bf16x8 w1 = ld8(reinterpret_cast<const bf16*>(a.conv_w) + (size_t)c * 4 + 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      w[e] = bf2f(w0[e]);
      w[8 + e] = bf2f(w1[e]);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(a.conv_w) + (size_t)c * 4 + 4 * q);
#pragma unroll
      for (int e = 0; e < 4; ++e) w[4 * q + e] = v[e];
    }
  }
  const T* cb = reinterpret_cast<const T*>(a.conv_b);
#pragma unroll
  for (int e = 0; e < 4; ++e) bias[e] = to_f32(cb[c + e]);
  bf16* ohi;
  bf16* olo;
  int ld, col;
  if (c < di) { ohi = a.x_hi; olo = a.x_lo; ld = di; col = c; }
  else if (c < di + gn) { ohi = a.B_hi; olo = a.B_lo; ld = gn; col = c - di; }
  else { ohi = a.C_hi; olo = a.C_lo; ld = gn; col = c - di - gn; }
#pragma unroll
  for (int u = 0; u < CONV_TT; ++u) {
    if (t0 + u >= a.T) break;
    bf16x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = bias[e];
#pragma unroll
      for (int j = 0; j < 4; ++j) v += w[4 * e + j] * in[u + j][e];
      v = silu(v);
      h[e] = f2bf(v);
      l[e] = f2bf(v - bf2f(h[e]));
    }
    const size_t o = ((size_t)b * a.T + t0 + u) * ld + col;
    *reinterpret_cast<bf16x4*>(ohi + o) = h;
    if (olo) *reinterpret_cast<bf16x4*>(olo + o) = l;
  }
}

// Vectorised causal conv: a thread owns 4 consecutive channels of one request and walks its
// T tokens in order with the last 8 inputs in registers, so zx is read once.  Needs the xBC and
// dt parts of a zx row 16-byte aligned (checked by the launcher).
template <typename T>
__global__ void __launch_bounds__(256) conv_split4_kernel(ConvArgs a) {
  const int di = a.H * a.P, gn = a.G * a.N, cdim = di + 2 * gn;
  const int dproj = 2 * di + 2 * gn + a.H;
  const int b = blockIdx.y;
  const int c = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (c >= cdim + a.H) return;
  const float* zrow = a.zxbcdt + (size_t)b * a.T * dproj;
  if (c >= cdim) {                                   // dt = softplus(dt_raw + dt_bias), 4 heads
    const int hh = c - cdim;
    for (int t = 0; t < a.T; ++t) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(zrow + (size_t)t * dproj + 2 * di + 2 * gn + hh);
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = softplus(v[e] + a.dt_bias[hh + e]);
      *reinterpret_cast<f32x4*>(a.dt + ((size_t)b * a.T + t) * a.H + hh) = o;
    }
    return;
  }
  const T* cw = reinterpret_cast<const T*>(a.conv_w);
  const T* cb = reinterpret_cast<const T*>(a.conv_b);
  // taps right-aligned in an 8-wide window: wp[j] multiplies the input 7 - j tokens back
  float wp[8][4], bias[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    bias[e] = to_f32(cb[c + e]);
#pragma unroll
    for (int j = 0; j < 8; ++j) wp[j][e] = j >= 8 - a.K ? to_f32(cw[(size_t)(c + e) * a.K + j - (8 - a.K)]) : 0.f;
  }
  f32x4 hist[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) hist[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16* ohi;
  bf16* olo;
  int ld, col;
  if (c < di) { ohi = a.x_hi; olo = a.x_lo; ld = di; col = c; }
  else if (c < di + gn) { ohi = a.B_hi; olo = a.B_lo; ld = gn; col = c - di; }
  else { ohi = a.C_hi; olo = a.C_lo; ld = gn; col = c - di - gn; }
  for (int t = 0; t < a.T; ++t) {
#pragma unroll
    for (int j = 0; j < 7; ++j) hist[j] = hist[j + 1];
    hist[7] = *reinterpret_cast<const f32x4*>(zrow + (size_t)t * dproj + di + c);
    bf16x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = bias[e];
#pragma unroll
      for (int j = 0; j < 8; ++j) v += wp[j][e] * hist[j][e];
      v = silu(v);
      h[e] = f2bf(v);
      l[e] = f2bf(v - bf2f(h[e]));
    }
    const size_t o = ((size_t)b * a.T + t) * ld + col;
    *reinterpret_cast<bf16x4*>(ohi + o) = h;
    if (olo) *reinterpret_cast<bf16x4*>(olo + o) = l;
  }
}

// One workgroup per (row, group); 8 elements per thread and step.  VEC: y and z rows can be
// read as 16-byte vectors.  NR > 0 (with VEC): the group fits in NR chunks of 8 per thread and is
// gated once, kept in registers between the sum of squares and the scaling pass (chunks past the
// group's end load its first chunk and count as zero); NR == 0: the second pass re-reads y and z.
template <bool VEC, int NR>
__global__ void __launch_bounds__(256) gated_rmsnorm_kernel(const float* y, const float* z, int z_ld,
                                                            const float* w, int n, int G, float eps,
                                                            bf16* hi, bf16* lo) {
  __shared__ float red[4];
  const size_t row = blockIdx.x / G;
  const int gi = blockIdx.x % G, gs = n / G;
  const float* yr = y + row * n + (size_t)gi * gs;
  const float* zr = z + row * z_ld + (size_t)gi * gs;
  auto gated8 = [&](int i, float (&v)[8]) {
    float zz[8];
    if constexpr (VEC) {
      load8(yr + i, v);
      load8(zr + i, zz);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] = yr[i + e];
        zz[e] = zr[i + e];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] *= silu(zz[e]);
  };
  if constexpr (NR > 0) {
    float v[NR][8], zz[NR][8];
#pragma unroll
    for (int c = 0; c < NR; ++c) {
      const int i = (threadIdx.x + c * 256) * 8, ic = i < gs ? i : 0;
      load8(yr + ic, v[c]);
      load8(zr + ic, zz[c]);
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NR; ++c) {
      const bool in = (threadIdx.x + c * 256) * 8 < gs;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[c][e] *= silu(zz[c][e]);
        ss += in ? v[c][e] * v[c][e] : 0.f;
      }
    }
    ss = block_sum(ss, red);
    const float r = rsqrtf(ss / gs + eps);
#pragma unroll
    for (int c = 0; c < NR; ++c) {
      const int i = (threadIdx.x + c * 256) * 8;
      if (i >= gs) break;
      float g[8];
      load8(w + (size_t)gi * gs + i, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = v[c][e] * r * g[e];
      put8(hi, lo, row * n + (size_t)gi * gs + i, v[c]);
    }
    return;
  }
  float ss = 0.f;
  for (int i = threadIdx.x * 8; i < gs; i += blockDim.x * 8) {
    float v[8];
    gated8(i, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  ss = block_sum(ss, red);
  const float r = rsqrtf(ss / gs + eps);
  for (int i = threadIdx.x * 8; i < gs; i += blockDim.x * 8) {
    float v[8], g[8];
    gated8(i, v);
    load8(w + (size_t)gi * gs + i, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * g[e];
    put8(hi, lo, row * n + (size_t)gi * gs + i, v);
  }
}

// Per-head RMSNorm of q and k, then rotate-half RoPE at position ctx_len + j; v heads are copied.
// One workgroup (4 waves) per token, for D a multiple of 8 with D/8 dividing 64 (D = 8 .. 512):
// a lane owns elements i0..i0+3 and i0 + D/2 .. i0 + D/2 + 3 of a head (16-byte loads, 8-byte
// plane stores), D/8 lanes per head.  The D/2 rotation angles of the token are computed once
// (in fp64, reduced modulo 2 pi, then fp32 sin/cos) by the first D/2 threads into LDS while the
// first heads load.
constexpr int QKR4_U = 4;

template <bool PLAN>
__global__ void __launch_bounds__(256) qk_norm_rope4_kernel(const float* qkv, const float* qw, const float* kw,
                                                            const int32_t* ctx_lens, int T, int Hq, int Hkv,
                                                            int D, float eps, double theta, bf16* q_hi,
                                                            bf16* q_lo, bf16* k_hi, bf16* k_lo, bf16* v_hi,
                                                            bf16* v_lo, AttnArgs plan, int plan_clear) {
  if constexpr (PLAN) {   // the first workgroup (dispatched first) builds the KV sweep's work list
    __shared__ WorklistLds<kWorklistFusedMax> wl;
    if (blockIdx.x == 0) {
      build_worklist<kWorklistFusedMax>(plan, plan_clear, wl);
      return;
    }
  }
  __shared__ float s_cs[256], s_sn[256];
  const int nh = Hq + 2 * Hkv;
  const int tok = PLAN ? blockIdx.x - 1 : blockIdx.x;
  const int b = tok / T, j = tok % T;
  const int half = D / 2, lph = D / 8, hpw = 64 / lph;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i0 = 4 * (lane % lph), hsub = lane / lph;
  const int hstep = 4 * hpw;                 // heads per workgroup pass
  const float* src_tok = qkv + (size_t)tok * nh * D;
  f32x4 x1[QKR4_U], x2[QKR4_U];
  auto load_heads = [&](int h0) {
#pragma unroll
    for (int u = 0; u < QKR4_U; ++u) {
      const int head = h0 + u * hstep + wave * hpw + hsub;
      const float* src = src_tok + (size_t)(head < nh ? head : 0) * D + i0;
      x1[u] = *reinterpret_cast<const f32x4*>(src);
      x2[u] = *reinterpret_cast<const f32x4*>(src + half);
    }
  };
  load_heads(0);
  for (int p = threadIdx.x; p < half; p += blockDim.x) {
    double phi = ((double)ctx_lens[b] + j) * pow(theta, -2.0 * (double)p / (double)D);
    const double two_pi = 6.283185307179586476925286766559;
    phi -= two_pi * rint(phi / two_pi);
    float sn, cs;
    sincosf((float)phi, &sn, &cs);
    s_cs[p] = cs;
    s_sn[p] = sn;
  }
  f32x4 gq1 = {0.f, 0.f, 0.f, 0.f}, gq2 = gq1;
  if (Hq > 0) {
    gq1 = *reinterpret_cast<const f32x4*>(qw + i0);
    gq2 = *reinterpret_cast<const f32x4*>(qw + half + i0);
  }
  const f32x4 gk1 = *reinterpret_cast<const f32x4*>(kw + i0), gk2 = *reinterpret_cast<const f32x4*>(kw + half + i0);
  __syncthreads();
  float cs[4], sn[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    cs[e] = s_cs[i0 + e];
    sn[e] = s_sn[i0 + e];
  }
  for (int h0 = 0; h0 < nh; h0 += QKR4_U * hstep) {
    if (h0) load_heads(h0);
#pragma unroll
    for (int u = 0; u < QKR4_U; ++u) {
      const int head = h0 + u * hstep + wave * hpw + hsub;
      // sum of squares over the head's D/8 lanes (every lane takes part in the exchange)
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) ss += x1[u][e] * x1[u][e] + x2[u][e] * x2[u][e];
      for (int off = lph / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      if (head >= nh) continue;
      float o1[4], o2[4];
      bf16 *hi, *lo;
      size_t o;
      if (head >= Hq + Hkv) {                  // v heads: copy
        o = ((size_t)tok * Hkv + (head - Hq - Hkv)) * D;
        hi = v_hi;
        lo = v_lo;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o1[e] = x1[u][e];
          o2[e] = x2[u][e];
        }
      } else {
        const bool isq = head < Hq;
        const float r = rsqrtf(ss / D + eps);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a1 = x1[u][e] * r * (isq ? gq1[e] : gk1[e]), a2 = x2[u][e] * r * (isq ? gq2[e] : gk2[e]);
          o1[e] = a1 * cs[e] - a2 * sn[e];
          o2[e] = a2 * cs[e] + a1 * sn[e];
        }
        hi = isq ? q_hi : k_hi;
        lo = isq ? q_lo : k_lo;
        o = isq ? ((size_t)tok * Hq + head) * D : ((size_t)tok * Hkv + (head - Hq)) * D;
      }
      bf16x4 h1, l1, h2, l2;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        h1[e] = f2bf(o1[e]);
        l1[e] = f2bf(o1[e] - bf2f(h1[e]));
        h2[e] = f2bf(o2[e]);
        l2[e] = f2bf(o2[e] - bf2f(h2[e]));
      }
      *reinterpret_cast<bf16x4*>(hi + o + i0) = h1;
      *reinterpret_cast<bf16x4*>(hi + o + half + i0) = h2;
      if (lo) {
        *reinterpret_cast<bf16x4*>(lo + o + i0) = l1;
        *reinterpret_cast<bf16x4*>(lo + o + half + i0) = l2;
      }
    }
  }
}

__global__ void split_kernel(const float* x, size_t n, bf16* hi, bf16* lo) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    put_planes(hi, lo, i, x[i]);
}

// h = SiLU(gate) * up for rows [gate | up] of width 2 ff, as bf16 hi/lo planes [rows, ff].
__global__ void __launch_bounds__(256) silu_mul_kernel(const float* gu, int ff, bf16* hi, bf16* lo) {
  const size_t row = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= ff) return;
  const float g = gu[row * 2 * ff + i], u = gu[row * 2 * ff + ff + i];
  const float v = silu(g) * u;
  const bf16 h = f2bf(v);
  hi[row * ff + i] = h;
  if (lo) lo[row * ff + i] = f2bf(v - bf2f(h));
}

// Appends the new rows [B*n, Hkv*D] (bf16 planes) of K and V at slot(ctx_len + i) of a paged
// cache.  Positions the table does not map, or page ids outside the pool, set a status bit and
// are skipped.
template <typename T>
__global__ void __launch_bounds__(256) kv_append_kernel(const bf16* k_hi, const bf16* k_lo, const bf16* v_hi,
                                                        const bf16* v_lo, int n, int row, const int32_t* pt,
                                                        int max_pages, int num_pages, int ps, const int32_t* lens,
                                                        T* kc, T* vc, int* status) {
  const int tok = blockIdx.x, b = tok / n, i = tok % n;
  const int L = lens[b];
  const int pos = L + i;
  const int pg = pos / ps;
  if (L < 0 || pg >= max_pages) {
    if (threadIdx.x == 0 && status) atomicOr(status, 2);
    return;
  }
  const int pid = pt[(size_t)b * max_pages + pg];
  if (pid < 0 || pid >= num_pages) {
    if (threadIdx.x == 0 && status) atomicOr(status, 1);
    return;
  }
  const size_t dst = ((size_t)pid * ps + pos % ps) * row, src = (size_t)tok * row;
  for (int e = threadIdx.x; e < row; e += blockDim.x) {
    float kv = bf2f(k_hi[src + e]), vv = bf2f(v_hi[src + e]);
    if (k_lo) kv += bf2f(k_lo[src + e]);
    if (v_lo) vv += bf2f(v_lo[src + e]);
    if constexpr (sizeof(T) == 2) {
      kc[dst + e] = f2bf(kv);
      vc[dst + e] = f2bf(vv);
    } else {
      kc[dst + e] = kv;
      vc[dst + e] = vv;
    }
  }
}

__global__ void zero_kernel(int* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

}  // namespace

hipError_t launch_rmsnorm_planes(const void* x, int x_bf16, const float* w, int rows, int n, float eps,
                                 bf16* out_hi, bf16* out_lo, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  // chunks of 8 per thread when the row is held in registers (0: two passes over the row)
  const int nr = n <= 2048 ? 1 : n <= 4096 ? 2 : n <= 8192 ? 4 : 0;
  auto launch = [&](auto xt, auto nrc) {
    using T = decltype(xt);
    hipLaunchKernelGGL((rmsnorm_kernel<T, decltype(nrc)::value>), dim3(rows), dim3(256), 0, s,
                       (const T*)x, w, n, eps, out_hi, out_lo);
  };
  auto by_type = [&](auto nrc) {
    if (x_bf16) launch(bf16{}, nrc);
    else launch(0.f, nrc);
  };
  switch (nr) {
    case 1: by_type(Int<1>{}); break;
    case 2: by_type(Int<2>{}); break;
    case 4: by_type(Int<4>{}); break;
    default: by_type(Int<0>{}); break;
  }
  return hipGetLastError();
}

hipError_t launch_conv_split(const ConvArgs& a, hipStream_t s) {
  const int di = a.H * a.P, gn = a.G * a.N;
  const int dproj = 2 * di + 2 * gn + a.H;
  const int total = di + 2 * gn + a.H;
  if (dproj % 4 == 0 && di % 4 == 0 && gn % 4 == 0 && a.H % 4 == 0 && a.K == 4) {
    dim3 grid((total / 4 + 255) / 256, a.B * ((a.T + CONV_TT - 1) / CONV_TT));
    if (a.w_bf16) hipLaunchKernelGGL(conv4_tok_kernel<bf16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(conv4_tok_kernel<float>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (dproj % 4 == 0 && di % 4 == 0 && gn % 4 == 0 && a.H % 4 == 0 && a.K <= 8) {
    dim3 grid((total / 4 + 255) / 256, a.B);
    if (a.w_bf16) hipLaunchKernelGGL(conv_split4_kernel<bf16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(conv_split4_kernel<float>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  dim3 grid((total + 255) / 256, a.B * a.T);
  if (a.w_bf16) hipLaunchKernelGGL(conv_split_kernel<bf16>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(conv_split_kernel<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gated_rmsnorm(const float* y, const float* z, int z_ld, const float* w, int rows, int n, int G,
                                float eps, bf16* out_hi, bf16* out_lo, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int gs = n / G;
  if (z_ld % 4 == 0 && gs % 4 == 0 && gs % 8 == 0 && gs <= 4096)
    hipLaunchKernelGGL((gated_rmsnorm_kernel<true, 2>), dim3(rows * G), dim3(256), 0, s, y, z, z_ld, w, n, G, eps, out_hi, out_lo);
  else if (z_ld % 4 == 0 && gs % 4 == 0 && gs % 8 == 0 && gs <= 8192)
    hipLaunchKernelGGL((gated_rmsnorm_kernel<true, 4>), dim3(rows * G), dim3(256), 0, s, y, z, z_ld, w, n, G, eps, out_hi, out_lo);
  else if (z_ld % 4 == 0 && gs % 4 == 0)
    hipLaunchKernelGGL((gated_rmsnorm_kernel<true, 0>), dim3(rows * G), dim3(256), 0, s, y, z, z_ld, w, n, G, eps, out_hi, out_lo);
  else
    hipLaunchKernelGGL((gated_rmsnorm_kernel<false, 0>), dim3(rows * G), dim3(256), 0, s, y, z, z_ld, w, n, G, eps, out_hi, out_lo);
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope(const float* qkv, const float* qw, const float* kw, const int32_t* ctx_lens, int B,
                               int T, int Hq, int Hkv, int D, float eps, double theta, bf16* q_hi, bf16* q_lo,
                               bf16* k_hi, bf16* k_lo, bf16* v_hi, bf16* v_lo, hipStream_t s, const AttnArgs* plan,
                               int plan_clear) {
  if (B * T <= 0) return hipSuccess;
  if (D < 8 || D % 8 || D > 512 || 64 % (D / 8)) return hipErrorInvalidValue;
  if (plan) {
    if (plan->B > kWorklistFusedMax) return hipErrorInvalidValue;
    hipLaunchKernelGGL(qk_norm_rope4_kernel<true>, dim3(B * T + 1), dim3(256), 0, s, qkv, qw, kw, ctx_lens, T,
                       Hq, Hkv, D, eps, theta, q_hi, q_lo, k_hi, k_lo, v_hi, v_lo, *plan, plan_clear);
  } else {
    hipLaunchKernelGGL(qk_norm_rope4_kernel<false>, dim3(B * T), dim3(256), 0, s, qkv, qw, kw, ctx_lens, T,
                       Hq, Hkv, D, eps, theta, q_hi, q_lo, k_hi, k_lo, v_hi, v_lo, AttnArgs{}, 0);
  }
  return hipGetLastError();
}

hipError_t launch_split_planes(const float* x, size_t n, bf16* hi, bf16* lo, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(split_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, n, hi, lo);
  return hipGetLastError();
}

hipError_t launch_silu_mul(const float* gu, int rows, int ff, bf16* hi, bf16* lo, hipStream_t s) {
  if (rows <= 0 || ff <= 0) return hipSuccess;
  hipLaunchKernelGGL(silu_mul_kernel, dim3((ff + 255) / 256, rows), dim3(256), 0, s, gu, ff, hi, lo);
  return hipGetLastError();
}

hipError_t launch_kv_append(const bf16* k_hi, const bf16* k_lo, const bf16* v_hi, const bf16* v_lo, int B, int n,
                            int Hkv, int D, const int32_t* page_table, int max_pages, int num_pages, int ps,
                            const int32_t* ctx_lens, void* k_cache, void* v_cache, int cache_bf16, int* status,
                            hipStream_t s) {
  if (B * n <= 0) return hipSuccess;
  if (cache_bf16)
    hipLaunchKernelGGL(kv_append_kernel<bf16>, dim3(B * n), dim3(256), 0, s, k_hi, k_lo, v_hi, v_lo, n, Hkv * D,
                       page_table, max_pages, num_pages, ps, ctx_lens, (bf16*)k_cache, (bf16*)v_cache, status);
  else
    hipLaunchKernelGGL(kv_append_kernel<float>, dim3(B * n), dim3(256), 0, s, k_hi, k_lo, v_hi, v_lo, n, Hkv * D,
                       page_table, max_pages, num_pages, ps, ctx_lens, (float*)k_cache, (float*)v_cache, status);
  return hipGetLastError();
}

hipError_t launch_zero_words(int* p, int n, hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace hspec
