// Normalisation, convolution and rotary kernels of the drafting step, plus small helpers.
// Each writes its result as bf16 planes ready to be MFMA operands (hi, and lo = rounding
// residual where the next contraction needs fp32-level accuracy).
#include "common.h"
#include "kernels.h"

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

template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const T* x, const float* w, int n, float eps,
                                                      bf16* hi, bf16* lo) {
  __shared__ float red[4];
  const size_t row = blockIdx.x;
  const T* xr = x + row * n;
  float ss = 0.f;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const float v = to_f32(xr[i]);
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float r = rsqrtf(ss / n + eps);
  for (int i = threadIdx.x; i < n; i += blockDim.x) put_planes(hi, lo, row * n + i, to_f32(xr[i]) * r * w[i]);
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

// One workgroup per (row, group).
__global__ void __launch_bounds__(256) gated_rmsnorm_kernel(const float* y, const float* z, int z_ld,
                                                            const float* w, int n, int G, float eps,
                                                            bf16* hi, bf16* lo) {
  __shared__ float red[4];
  const size_t row = blockIdx.x / G;
  const int gi = blockIdx.x % G, gs = n / G;
  const float* yr = y + row * n + (size_t)gi * gs;
  const float* zr = z + row * z_ld + (size_t)gi * gs;
  float ss = 0.f;
  for (int i = threadIdx.x; i < gs; i += blockDim.x) {
    const float v = yr[i] * silu(zr[i]);
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float r = rsqrtf(ss / gs + eps);
  for (int i = threadIdx.x; i < gs; i += blockDim.x)
    put_planes(hi, lo, row * n + (size_t)gi * gs + i, yr[i] * silu(zr[i]) * r * w[gi * gs + i]);
}

// One wave per (token, head) of q, k and v.  Lane i < D/2 owns the rotate-half pair (i, i + D/2).
__global__ void __launch_bounds__(64) qk_norm_rope_kernel(const float* qkv, const float* qw, const float* kw,
                                                          const int32_t* ctx_lens, int T, int Hq, int Hkv,
                                                          int D, float eps, double theta, bf16* q_hi,
                                                          bf16* q_lo, bf16* k_hi, bf16* k_lo, bf16* v_hi,
                                                          bf16* v_lo) {
  const int nh = Hq + 2 * Hkv;
  const int tok = blockIdx.x / nh, head = blockIdx.x % nh;
  const int b = tok / T, j = tok % T;
  const int lane = threadIdx.x, half = D / 2;
  const float* src = qkv + (size_t)tok * nh * D + (size_t)head * D;
  const bool act = lane < half;
  const float x1 = act ? src[lane] : 0.f, x2 = act ? src[lane + half] : 0.f;
  if (head >= Hq + Hkv) {                     // v: copy
    if (act) {
      const size_t o = ((size_t)tok * Hkv + (head - Hq - Hkv)) * D;
      put_planes(v_hi, v_lo, o + lane, x1);
      put_planes(v_hi, v_lo, o + lane + half, x2);
    }
    return;
  }
  const bool isq = head < Hq;
  const float* g = isq ? qw : kw;
  const float ss = wave_sum(x1 * x1 + x2 * x2);
  const float r = rsqrtf(ss / D + eps);
  const float a1 = act ? x1 * r * g[lane] : 0.f, a2 = act ? x2 * r * g[lane + half] : 0.f;
  // angle in fp64: pos * theta^(-2i/D), reduced modulo 2 pi before the fp32 sin/cos
  const double pos = (double)ctx_lens[b] + j;
  const double inv = pow(theta, -2.0 * (double)lane / (double)D);
  double phi = pos * inv;
  const double two_pi = 6.283185307179586476925286766559;
  phi -= two_pi * rint(phi / two_pi);
  float sn, cs;
  sincosf((float)phi, &sn, &cs);
  if (!act) return;
  const float o1 = a1 * cs - a2 * sn, o2 = a2 * cs + a1 * sn;
  bf16* hi = isq ? q_hi : k_hi;
  bf16* lo = isq ? q_lo : k_lo;
  const size_t o = isq ? ((size_t)tok * Hq + head) * D : ((size_t)tok * Hkv + (head - Hq)) * D;
  put_planes(hi, lo, o + lane, o1);
  put_planes(hi, lo, o + lane + half, o2);
}

__global__ void split_kernel(const float* x, size_t n, bf16* hi, bf16* lo) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    put_planes(hi, lo, i, x[i]);
}

__global__ void zero_kernel(int* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

}  // namespace

hipError_t launch_rmsnorm_planes(const void* x, int x_bf16, const float* w, int rows, int n, float eps,
                                 bf16* out_hi, bf16* out_lo, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (x_bf16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16>, dim3(rows), dim3(256), 0, s, (const bf16*)x, w, n, eps, out_hi, out_lo);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)x, w, n, eps, out_hi, out_lo);
  return hipGetLastError();
}

hipError_t launch_conv_split(const ConvArgs& a, hipStream_t s) {
  const int total = a.H * a.P + 2 * a.G * a.N + a.H;
  dim3 grid((total + 255) / 256, a.B * a.T);
  if (a.w_bf16) hipLaunchKernelGGL(conv_split_kernel<bf16>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(conv_split_kernel<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gated_rmsnorm(const float* y, const float* z, int z_ld, const float* w, int rows, int n, int G,
                                float eps, bf16* out_hi, bf16* out_lo, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(gated_rmsnorm_kernel, dim3(rows * G), dim3(256), 0, s, y, z, z_ld, w, n, G, eps, out_hi, out_lo);
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope(const float* qkv, const float* qw, const float* kw, const int32_t* ctx_lens, int B,
                               int T, int Hq, int Hkv, int D, float eps, double theta, bf16* q_hi, bf16* q_lo,
                               bf16* k_hi, bf16* k_lo, bf16* v_hi, bf16* v_lo, hipStream_t s) {
  if (B * T <= 0) return hipSuccess;
  hipLaunchKernelGGL(qk_norm_rope_kernel, dim3(B * T * (Hq + 2 * Hkv)), dim3(64), 0, s, qkv, qw, kw, ctx_lens, T,
                     Hq, Hkv, D, eps, theta, q_hi, q_lo, k_hi, k_lo, v_hi, v_lo);
  return hipGetLastError();
}

hipError_t launch_split_planes(const float* x, size_t n, bf16* hi, bf16* lo, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(split_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, n, hi, lo);
  return hipGetLastError();
}

hipError_t launch_zero_words(int* p, int n, hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace hspec
