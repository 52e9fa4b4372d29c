// Chunked SSD scan of the Mamba-2 selective recurrence from an injected initial state
// (H-Spec Sec. 3.3.1: the Mamba kernel starts from the projected last-token state and
// evaluates every draft position in one pass).
//
// Per head (scalar decay a_t = exp(dt_t A)), within a chunk with l_t = sum_{u<=t} dt_u A:
//   y_t = exp(l_t) C_t S_in^T + sum_{s<=t} exp(l_t - l_s) dt_s (C_t . B_s) x_s + D x_t
//   S_out = exp(l_end) S_in + sum_s exp(l_end - l_s) dt_s x_s (outer) B_s
// One wave owns one (request, head).  C S_in^T (16 x N x 64) and C B^T (16 x N x 16) run on
// v_mfma_f32_16x16x32_bf16; operands given as bf16 hi/lo planes use three products so fp32
// values survive.  The 16x16 decay-weighted mixing matrix and the x tile go through LDS and
// the intra-chunk product is done in fp32 on the VALU.  The chunk-local cumulative sum of
// dt*A is a 16-lane shuffle scan.  When the block fits one chunk and no final state is
// requested (ssd_scan_one), the initial state is read straight from global memory into MFMA
// fragments (as bf16 hi/lo planes, or as one fp16 plane multiplied with C rounded to fp16 on
// v_mfma_f32_16x16x32_f16); with the fp16 plane and heads in groups of 4 that share B and C
// (the drafting step), ssd_scan_grp runs those 4 heads in one workgroup, one wave each, and
// shares the C and C B^T work through LDS; otherwise (ssd_scan_kernel) the fp32 state lives
// in LDS between chunks.
#include "common.h"
#include "kernels.h"

namespace hspec {

namespace {

constexpr int P = 64;
constexpr int QMAX = 16;

template <int N>
struct ScanLds {
  static constexpr int XT = P * (QMAX + 1);          // x^T tile, fp32, padded rows
  static constexpr int MM = QMAX * (QMAX + 1);        // mixing matrix, fp32
  static constexpr int BT = N * (QMAX + 1);           // B^T tile, fp32
  static constexpr int ST = P * (N + 1);              // state, fp32, padded rows
  static constexpr int BYTES = 4 * (XT + MM + BT + ST);
};

__device__ __forceinline__ bf16x8 ld8_or0(const bf16* p, bool ok) { return ok ? ld8(p) : zero8(); }

__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const bf16 h = f2bf(v[e]);
    hi[e] = h;
    lo[e] = f2bf(v[e] - bf2f(h));
  }
}

// Intra-chunk term M x on v_mfma_f32_16x16x32_bf16: A = M (row t = lane % 16, k = s), B = x^T
// (k = s, column p = 16 pb + lane % 16); k = 16..31 are zero.  Both fp32 tiles enter as bf16
// hi/lo planes (three products).  Lane gets rows t = 4 (lane / 16) + i of column p, the layout
// of the state term.  M is zero for s > t and outside the chunk, x^T for s outside it.
__device__ __forceinline__ void mix_mfma(const float* Mm, const float* xT, int lane, f32x4 (&mx)[4]) {
  const int g4 = lane >> 4, l16 = lane & 15;
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = g4 < 2 ? Mm[l16 * (QMAX + 1) + 8 * g4 + e] : 0.f;
  bf16x8 mh, ml;
  split8(v, mh, ml);
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = g4 < 2 ? xT[(16 * pb + l16) * (QMAX + 1) + 8 * g4 + e] : 0.f;
    bf16x8 xh, xl;
    split8(v, xh, xl);
    mx[pb] = mma16(mh, xh, f32x4{0.f, 0.f, 0.f, 0.f});
    mx[pb] = mma16(ml, xh, mx[pb]);
    mx[pb] = mma16(mh, xl, mx[pb]);
  }
}

template <int N>
__global__ void __launch_bounds__(64) ssd_scan_kernel(ScanArgs a) {
  constexpr int NS = (N + 31) / 32;
  using LD = ScanLds<N>;
  extern __shared__ __align__(16) float sm[];
  float* xT = sm;                       // [P][QMAX+1]
  float* Mm = xT + LD::XT;              // [QMAX][QMAX+1]
  float* Bt = Mm + LD::MM;              // [N][QMAX+1]
  float* S = Bt + LD::BT;               // [P][N+1]

  const int H = a.H, T = a.T, G = a.G;
  const int b = blockIdx.x / H, h = blockIdx.x % H;
  const int grp = h / (H / G);
  const int lane = threadIdx.x, g4 = lane >> 4, l16 = lane & 15;
  const float Ah = a.A_is_log ? -__expf(a.A[h]) : a.A[h], Dh = a.Dskip[h];
  const size_t s0_off = ((size_t)b * H + h) * P * N;

  // S0 into LDS in 16-byte pieces (8 elements of a row), every load of a round issued before
  // its first LDS write (two rounds at N = 128 to bound the registers)
  {
    constexpr int PR = N / 8, PER = P * PR / 64, RND = PER > 8 ? PER / 2 : PER;
#pragma unroll
    for (int r0 = 0; r0 < PER; r0 += RND) {
      bf16x8 hv[RND], lv[RND];
      f16x8 fv[RND];
#pragma unroll
      for (int j = 0; j < RND; ++j) {
        const int q = (r0 + j) * 64 + lane, p = q / PR, n0 = (q % PR) * 8;
        const size_t off = s0_off + (size_t)p * N + n0;
        if (a.S0_h16) {
          fv[j] = *reinterpret_cast<const f16x8*>(a.S0_h16 + off);
        } else {
          hv[j] = ld8_or0(a.S0_hi + off, a.S0_hi != nullptr);
          lv[j] = ld8_or0(a.S0_lo + off, a.S0_lo != nullptr);
        }
      }
#pragma unroll
      for (int j = 0; j < RND; ++j) {
        const int q = (r0 + j) * 64 + lane, p = q / PR, n0 = (q % PR) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          S[p * (N + 1) + n0 + e] = a.S0_h16 ? (float)fv[j][e] : bf2f(hv[j][e]) + bf2f(lv[j][e]);
      }
    }
  }
  __syncthreads();

  // A chunk's global inputs (dt, the x tile, the C and B fragments) come into registers one
  // chunk ahead: the next chunk's loads are in flight while this one is computed.
  struct ChunkIn {
    float dtv;
    bf16x8 xh0, xh1, xl0, xl1;
    bf16x8 cf[NS], cfl[NS], bfr[NS], bfl[NS];
  };
  auto load_chunk = [&](int c0, ChunkIn& r) {
    const int Qc = max(0, min(a.chunk, T - c0));   // 0 past the last chunk: nothing is read
    r.dtv = l16 < Qc ? a.dt[(size_t)(b * T + c0 + l16) * a.dt_ld + h] : 0.f;
    // x tile: lane holds x[t = lane / 4][p = 16 (lane % 4) .. + 15], zero past the chunk
    const int xt = lane >> 2, xp = 16 * (lane & 3);
    const bool xok = xt < Qc;
    const size_t xoff = (size_t)(b * T + c0 + xt) * a.x_ld + (size_t)h * P + xp;
    r.xh0 = ld8_or0(a.x_hi + xoff, xok);
    r.xh1 = ld8_or0(a.x_hi + xoff + 8, xok);
    r.xl0 = a.x_lo ? ld8_or0(a.x_lo + xoff, xok) : zero8();
    r.xl1 = a.x_lo ? ld8_or0(a.x_lo + xoff + 8, xok) : zero8();
    // C (A operand, rows t) and B (B operand, columns s) fragments over n
    const size_t tok_t = (size_t)(b * T + c0 + l16) * a.bc_ld + (size_t)grp * N;
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) {
      const int n = 32 * ns + 8 * g4;
      const bool ok = l16 < Qc && n < N;
      r.cf[ns] = ld8_or0(a.C_hi + tok_t + n, ok);
      r.cfl[ns] = a.C_lo ? ld8_or0(a.C_lo + tok_t + n, ok) : zero8();
      r.bfr[ns] = ld8_or0(a.B_hi + tok_t + n, ok);
      r.bfl[ns] = a.B_lo ? ld8_or0(a.B_lo + tok_t + n, ok) : zero8();
    }
  };
  ChunkIn nx;
  load_chunk(0, nx);

  for (int c0 = 0; c0 < T; c0 += a.chunk) {
    const int Qc = min(a.chunk, T - c0);
    const ChunkIn cur = nx;
    load_chunk(c0 + a.chunk, nx);
    const float dtv = cur.dtv;
    // the inclusive cumulative sum of dt*A over the chunk (lanes 0..15)
    float cum = dtv * Ah;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float v = __shfl_up(cum, off, 16);
      if (l16 >= off) cum += v;
    }
    // x^T tile in LDS
    {
      const int xt = lane >> 2, xp = 16 * (lane & 3);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xT[(xp + e) * (QMAX + 1) + xt] = bf2f(cur.xh0[e]) + bf2f(cur.xl0[e]);
        xT[(xp + 8 + e) * (QMAX + 1) + xt] = bf2f(cur.xh1[e]) + bf2f(cur.xl1[e]);
      }
    }
    const bf16x8 *cf = cur.cf, *cfl = cur.cfl, *bfr = cur.bfr, *bfl = cur.bfl;
    // state term C S^T: lane gets rows t = 4 g4 + i, column p = 16 pb + l16
    f32x4 ys[4];
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) {
      ys[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int p = 16 * pb + l16;
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) {
        const int n = 32 * ns + 8 * g4;
        bf16x8 sh, sl;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = n + e < N ? S[p * (N + 1) + n + e] : 0.f;
        split8(v, sh, sl);
        ys[pb] = mma16(cf[ns], sh, ys[pb]);
        if (a.C_lo) ys[pb] = mma16(cfl[ns], sh, ys[pb]);
        ys[pb] = mma16(cf[ns], sl, ys[pb]);
      }
    }
    // C B^T: lane gets rows t = 4 g4 + i, column s = l16
    f32x4 cb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) {
      cb = mma16(cf[ns], bfr[ns], cb);
      if (a.C_lo) cb = mma16(cfl[ns], bfr[ns], cb);
      if (a.B_lo) cb = mma16(cf[ns], bfl[ns], cb);
    }
    const float ell_s = __shfl(cum, l16);            // l_s for this lane's column s
    const float dt_s = __shfl(dtv, l16);
    float ell_t[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 4 * g4 + i;
      ell_t[i] = __shfl(cum, t);
      const bool ok = l16 <= t && t < Qc;
      Mm[t * (QMAX + 1) + l16] = ok ? cb[i] * __expf(ell_t[i] - ell_s) * dt_s : 0.f;
    }
    // B^T tile for the state update, Bt[n][s], from the B fragments already in registers
    // (token s = lane % 16, zero past the chunk)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int n = 32 * ns + 8 * g4 + e;
        if (n < N) Bt[n * (QMAX + 1) + l16] = bf2f(bfr[ns][e]) + bf2f(bfl[ns][e]);
      }
    __syncthreads();
    // y = exp(l_t) (C S^T) + M x + D x, M x on MFMA
    f32x4 mx[4];
    mix_mfma(Mm, xT, lane, mx);
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) {
      const int p = 16 * pb + l16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 4 * g4 + i;
        if (t >= Qc) continue;
        const float acc = __expf(ell_t[i]) * ys[pb][i] + Dh * xT[p * (QMAX + 1) + t] + mx[pb][i];
        a.y[(size_t)(b * T + c0 + t) * H * P + (size_t)h * P + p] = acc;
      }
    }
    {
      // S <- exp(l_end) S + (W X) B on v_mfma_f32_32x32x16_bf16: A = W X (row p, k = s) with
      // W X [p][s] = exp(l_end - l_s) dt_s x_s[p], B = the B tile (k = s, column n), the
      // accumulator the decayed state in the 32 x 32 block layout (lane holds rows
      // 8 (i / 4) + 4 (lane / 32) + i % 4 of column lane % 32), read from and written back to
      // LDS by the same lane.  fp32 operands as bf16 hi/lo planes (three products).
      const float ell_end = __shfl(cum, Qc - 1);
      const float dec = __expf(ell_end);
      const int r32 = lane & 31, h2 = lane >> 5;
      float wv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sx = 8 * h2 + e;
        const float w = __shfl(dtv, sx) * __expf(ell_end - __shfl(cum, sx));
        wv[e] = sx < Qc ? w : 0.f;
      }
      bf16x8 wh[2], wl[2];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = wv[e] * xT[(32 * pb + r32) * (QMAX + 1) + 8 * h2 + e];
        split8(v, wh[pb], wl[pb]);
      }
#pragma unroll
      for (int nb = 0; nb < (N + 31) / 32; ++nb) {
        const int n = 32 * nb + r32;
        const bool nok = n < N;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = nok ? Bt[n * (QMAX + 1) + 8 * h2 + e] : 0.f;
        bf16x8 bh, bl;
        split8(v, bh, bl);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          f32x16 acc;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int p = 32 * pb + 8 * (i / 4) + 4 * h2 + (i % 4);
            acc[i] = nok ? dec * S[p * (N + 1) + n] : 0.f;
          }
          acc = mma32(wh[pb], bh, acc);
          acc = mma32(wl[pb], bh, acc);
          acc = mma32(wh[pb], bl, acc);
          if (nok) {
#pragma unroll
            for (int i = 0; i < 16; ++i) S[(32 * pb + 8 * (i / 4) + 4 * h2 + (i % 4)) * (N + 1) + n] = acc[i];
          }
        }
      }
    }
    __syncthreads();
  }

  if (a.S_final) {
    // 16-byte stores where the caller's buffer allows them
    const bool vec = (reinterpret_cast<uintptr_t>(a.S_final) & 15) == 0;
    for (int q = lane; q < P * N / 4; q += 64) {
      const int p = q / (N / 4), n0 = (q % (N / 4)) * 4;
      const float* sr = S + p * (N + 1) + n0;
      float* dst = a.S_final + s0_off + (size_t)p * N + n0;
      if (vec) {
        *reinterpret_cast<f32x4*>(dst) = f32x4{sr[0], sr[1], sr[2], sr[3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[e] = sr[e];
      }
    }
  }
}

// The block in one chunk and no final state (every drafting step): the same arithmetic as
// ssd_scan_kernel<N, false>, with every global load of the wave (dt, the x tile, the B and C
// fragments, all initial-state fragments) issued before the first is used, so that a wave
// waits for memory once instead of once per state fragment.
template <int N, bool H16>
__global__ void __launch_bounds__(64) ssd_scan_one(ScanArgs a) {
  constexpr int NS = (N + 31) / 32;
  __shared__ float xT[P * (QMAX + 1)];   // x^T tile, fp32, padded rows
  __shared__ float Mm[QMAX * (QMAX + 1)];

  const int H = a.H, T = a.T, G = a.G;
  const int b = blockIdx.x / H, h = blockIdx.x % H;
  const int grp = h / (H / G);
  const int lane = threadIdx.x, g4 = lane >> 4, l16 = lane & 15;
  const size_t s0_off = ((size_t)b * H + h) * P * N;

  // ---- loads, in order of use
  const float dtv = l16 < T ? a.dt[(size_t)(b * T + l16) * a.dt_ld + h] : 0.f;
  // x tile: lane holds x[t = lane / 4][p = 16 (lane % 4) .. + 15]
  const int xt = lane >> 2, xp = 16 * (lane & 3);
  const bool xok = xt < T;
  const size_t xoff = (size_t)(b * T + xt) * a.x_ld + (size_t)h * P + xp;
  const bf16x8 xh0 = ld8_or0(a.x_hi + xoff, xok), xh1 = ld8_or0(a.x_hi + xoff + 8, xok);
  const bf16x8 xl0 = a.x_lo ? ld8_or0(a.x_lo + xoff, xok) : zero8();
  const bf16x8 xl1 = a.x_lo ? ld8_or0(a.x_lo + xoff + 8, xok) : zero8();
  // C (A operand, rows t) and B (B operand, columns s) fragments over n
  bf16x8 cf[NS], cfl[NS], bfr[NS], bfl[NS];
  const size_t tok_t = (size_t)(b * T + l16) * a.bc_ld + (size_t)grp * N;
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) {
    const int n = 32 * ns + 8 * g4;
    const bool ok = l16 < T && n < N;
    cf[ns] = ld8_or0(a.C_hi + tok_t + n, ok);
    cfl[ns] = a.C_lo ? ld8_or0(a.C_lo + tok_t + n, ok) : zero8();
    bfr[ns] = ld8_or0(a.B_hi + tok_t + n, ok);
    bfl[ns] = a.B_lo ? ld8_or0(a.B_lo + tok_t + n, ok) : zero8();
  }
  // initial state as B operand of C S^T: column p = 16 pb + l16, n = 32 ns + 8 g4 ..  (H16: one
  // fp16 plane, multiplied with C rounded to fp16; otherwise bf16 hi/lo planes)
  bf16x8 sh[4][H16 ? 1 : NS], sl[4][H16 ? 1 : NS];
  f16x8 s16[4][H16 ? NS : 1];
#pragma unroll
  for (int pb = 0; pb < 4; ++pb)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) {
      const int n = 32 * ns + 8 * g4;
      const size_t off = s0_off + (size_t)(16 * pb + l16) * N + n;
      if constexpr (H16) {
        s16[pb][ns] = n < N ? *reinterpret_cast<const f16x8*>(a.S0_h16 + off) : f16x8{};
      } else {
        const bool ok = a.S0_hi != nullptr && n < N;
        sh[pb][ns] = ld8_or0(a.S0_hi + off, ok);
        sl[pb][ns] = a.S0_lo != nullptr ? ld8_or0(a.S0_lo + off, ok) : zero8();
      }
    }
  const float Ah = a.A_is_log ? -__expf(a.A[h]) : a.A[h], Dh = a.Dskip[h];

  // ---- inclusive cumulative sum of dt*A over the chunk (lanes 0..15)
  float cum = dtv * Ah;
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) {
    const float v = __shfl_up(cum, off, 16);
    if (l16 >= off) cum += v;
  }
  // ---- x^T tile in LDS
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    xT[(xp + e) * (QMAX + 1) + xt] = bf2f(xh0[e]) + bf2f(xl0[e]);
    xT[(xp + 8 + e) * (QMAX + 1) + xt] = bf2f(xh1[e]) + bf2f(xl1[e]);
  }
  // ---- C B^T: lane gets rows t = 4 g4 + i, column s = l16
  f32x4 cb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) {
    cb = mma16(cf[ns], bfr[ns], cb);
    if (a.C_lo) cb = mma16(cfl[ns], bfr[ns], cb);
    if (a.B_lo) cb = mma16(cf[ns], bfl[ns], cb);
  }
  // ---- state term C S^T: lane gets rows t = 4 g4 + i, column p = 16 pb + l16
  f32x4 ys[4];
  if constexpr (H16) {
    f16x8 c16[NS];   // C (hi + lo) rounded once to fp16
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
#pragma unroll
      for (int e = 0; e < 8; ++e) c16[ns][e] = (_Float16)(bf2f(cf[ns][e]) + bf2f(cfl[ns][e]));
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) {
      ys[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) ys[pb] = mma16h(c16[ns], s16[pb][ns], ys[pb]);
    }
  } else {
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) {
      ys[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) {
        ys[pb] = mma16(cf[ns], sh[pb][ns], ys[pb]);
        if (a.C_lo) ys[pb] = mma16(cfl[ns], sh[pb][ns], ys[pb]);
        if (a.S0_lo) ys[pb] = mma16(cf[ns], sl[pb][ns], ys[pb]);
      }
    }
  }
  // ---- decay-weighted mixing matrix M[t][s] = (C_t . B_s) exp(l_t - l_s) dt_s for s <= t
  const float ell_s = __shfl(cum, l16);
  const float dt_s = __shfl(dtv, l16);
  float ell_t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = 4 * g4 + i;
    ell_t[i] = __shfl(cum, t);
    const bool ok = l16 <= t && t < T;
    Mm[t * (QMAX + 1) + l16] = ok ? cb[i] * __expf(ell_t[i] - ell_s) * dt_s : 0.f;
  }
  __syncthreads();
  // ---- y = exp(l_t) (C S^T) + M x + D x, M x on MFMA (every entry of both tiles is written
  // above: M is zero for s > t and past the block, x^T for s past it)
  f32x4 mx[4];
  mix_mfma(Mm, xT, lane, mx);
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) {
    const int p = 16 * pb + l16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 4 * g4 + i;
      const float acc = __expf(ell_t[i]) * ys[pb][i] + Dh * xT[p * (QMAX + 1) + t] + mx[pb][i];
      if (t < T) a.y[(size_t)(b * T + t) * H * P + (size_t)h * P + p] = acc;
    }
  }
}

// The drafting step's case (one chunk, no final state, S0 as one fp16 plane) with HW waves per
// workgroup, one per head, for HW heads of one request that read the same B and C.  Each wave
// loads only its own head's S0, dt and x, so it holds a third fewer registers than
// ssd_scan_one and more waves stay resident; wave w loads the w-th (mod HW) 32-wide slices of
// C and B, rounds its C slice to fp16 into LDS and leaves its part of C B^T there, and every
// wave adds the parts in slice order.  The arithmetic is ssd_scan_one<N, true>'s: C S0^T as
// sum over slices of fp16 products, C B^T from the hi/lo planes, the rest unchanged.
constexpr int SCAN_HW = 4;
template <int N>
__global__ void __launch_bounds__(64 * SCAN_HW) __attribute__((amdgpu_waves_per_eu(4))) ssd_scan_grp(ScanArgs a) {
  constexpr int NS = (N + 31) / 32;
  constexpr int CP = N + 8;   // fp16 C row pitch (16 bytes of padding)
  __shared__ float xT_all[SCAN_HW][P * (QMAX + 1)];
  __shared__ float Mm_all[SCAN_HW][QMAX * (QMAX + 1)];
  __shared__ __align__(16) _Float16 c16s[QMAX * CP];   // C rounded to fp16, rows t
  __shared__ f32x4 cbp[NS][64];                         // parts of C B^T, one per slice

  const int H = a.H, T = a.T, G = a.G;
  // (the wave index made visibly uniform: the head's A, D and offsets become scalar values)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g4 = lane >> 4, l16 = lane & 15;
  const int hpb = H / SCAN_HW;                          // workgroups per request
  const int b = blockIdx.x / hpb, h = (blockIdx.x % hpb) * SCAN_HW + wave;
  const int grp = h / (H / G);                          // the same for the workgroup's heads
  const size_t s0_off = ((size_t)b * H + h) * P * N;
  float* xT = xT_all[wave];
  float* Mm = Mm_all[wave];

  // ---- loads, in order of use: dt and x of this head, this wave's slices of C and B, S0.
  // Lanes past the block read token 0 (no branch around a load, whose merged value would
  // have to arrive before the next load is issued) and drop the value where it is used.
  const bool tok_ok = l16 < T;
  const float dt_raw = a.dt[(size_t)(b * T + (tok_ok ? l16 : 0)) * a.dt_ld + h];
  const int xt = lane >> 2, xp = 16 * (lane & 3);
  const bool xok = xt < T;
  const size_t xoff = (size_t)(b * T + (xok ? xt : 0)) * a.x_ld + (size_t)h * P + xp;
  const bf16x8 xh0 = ld8(a.x_hi + xoff), xh1 = ld8(a.x_hi + xoff + 8);
  // (lo planes: the hi plane is read in their place when there is none, and dropped)
  const bf16* x_lo = a.x_lo ? a.x_lo : a.x_hi;
  const bf16x8 xl0 = ld8(x_lo + xoff), xl1 = ld8(x_lo + xoff + 8);
  const size_t tok_t = (size_t)(b * T + (tok_ok ? l16 : 0)) * a.bc_ld + (size_t)grp * N;
  constexpr int NSW = (NS + SCAN_HW - 1) / SCAN_HW;    // slices per wave
  bf16x8 cf[NSW], cfl[NSW], bfr[NSW], bfl[NSW];
#pragma unroll
  for (int kk = 0; kk < NSW; ++kk) {
    const int ns = wave + SCAN_HW * kk;
    const int n = 32 * ns + 8 * g4;
    const int nc = ns < NS && n < N ? n : 0;   // (in range; the value is dropped below)
    cf[kk] = ld8(a.C_hi + tok_t + nc);
    cfl[kk] = ld8((a.C_lo ? a.C_lo : a.C_hi) + tok_t + nc);
    bfr[kk] = ld8(a.B_hi + tok_t + nc);
    bfl[kk] = ld8((a.B_lo ? a.B_lo : a.B_hi) + tok_t + nc);
  }
  f16x8 s16[4][NS];
#pragma unroll
  for (int pb = 0; pb < 4; ++pb)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) {
      const int n = 32 * ns + 8 * g4;
      s16[pb][ns] = n < N ? *reinterpret_cast<const f16x8*>(a.S0_h16 + s0_off + (size_t)(16 * pb + l16) * N + n)
                          : f16x8{};
    }
  const float Ah = a.A_is_log ? -__expf(a.A[h]) : a.A[h], Dh = a.Dskip[h];

  // ---- this wave's C slices (fp16, rows t = l16) and parts of C B^T into LDS
#pragma unroll
  for (int kk = 0; kk < NSW; ++kk) {
    const int ns = wave + SCAN_HW * kk;
    if (ns < NS) {   // (uniform: ns depends on the wave only)
      // the C and B rows of tokens past the block, and columns past N, are zero
      const bool ok = tok_ok && 32 * ns + 8 * g4 < N;
      const bf16x8 cv = ok ? cf[kk] : zero8(), cvl = ok && a.C_lo ? cfl[kk] : zero8();
      const bf16x8 bv = ok ? bfr[kk] : zero8(), bvl = ok && a.B_lo ? bfl[kk] : zero8();
      f32x4 part = {0.f, 0.f, 0.f, 0.f};
      part = mma16(cv, bv, part);
      if (a.C_lo) part = mma16(cvl, bv, part);
      if (a.B_lo) part = mma16(cv, bvl, part);
      cbp[ns][lane] = part;
      f16x8 c;
#pragma unroll
      for (int e = 0; e < 8; ++e) c[e] = (_Float16)(bf2f(cv[e]) + bf2f(cvl[e]));
      if (32 * ns + 8 * g4 < N) *reinterpret_cast<f16x8*>(c16s + l16 * CP + 32 * ns + 8 * g4) = c;
    }
  }
  // ---- inclusive cumulative sum of dt*A over the chunk (lanes 0..15)
  const float dtv = tok_ok ? dt_raw : 0.f;
  float cum = dtv * Ah;
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) {
    const float v = __shfl_up(cum, off, 16);
    if (l16 >= off) cum += v;
  }
  // ---- x^T tile of this head in LDS (zero past the block)
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    xT[(xp + e) * (QMAX + 1) + xt] = xok ? bf2f(xh0[e]) + (a.x_lo ? bf2f(xl0[e]) : 0.f) : 0.f;
    xT[(xp + 8 + e) * (QMAX + 1) + xt] = xok ? bf2f(xh1[e]) + (a.x_lo ? bf2f(xl1[e]) : 0.f) : 0.f;
  }
  __syncthreads();   // C slices and parts of C B^T from every wave
  // ---- C B^T: lane gets rows t = 4 g4 + i, column s = l16 (parts added in slice order)
  f32x4 cb = cbp[0][lane];
#pragma unroll
  for (int ns = 1; ns < NS; ++ns) cb += cbp[ns][lane];
  // ---- state term C S^T: lane gets rows t = 4 g4 + i, column p = 16 pb + l16
  f32x4 ys[4];
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) ys[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) {
    const int n = 32 * ns + 8 * g4;   // (columns past N, N = 16: zero, as S0 is there)
    const f16x8 c = n < N ? *reinterpret_cast<const f16x8*>(c16s + l16 * CP + n) : f16x8{};
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) ys[pb] = mma16h(c, s16[pb][ns], ys[pb]);
  }
  // ---- decay-weighted mixing matrix M[t][s] = (C_t . B_s) exp(l_t - l_s) dt_s for s <= t
  const float ell_s = __shfl(cum, l16);
  const float dt_s = __shfl(dtv, l16);
  float ell_t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = 4 * g4 + i;
    ell_t[i] = __shfl(cum, t);
    const bool ok = l16 <= t && t < T;
    Mm[t * (QMAX + 1) + l16] = ok ? cb[i] * __expf(ell_t[i] - ell_s) * dt_s : 0.f;
  }
  __syncthreads();   // (each wave reads only its own tiles; one barrier for the LDS writes)
  // ---- y = exp(l_t) (C S^T) + M x + D x
  f32x4 mx[4];
  mix_mfma(Mm, xT, lane, mx);
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) {
    const int p = 16 * pb + l16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = 4 * g4 + i;
      const float acc = __expf(ell_t[i]) * ys[pb][i] + Dh * xT[p * (QMAX + 1) + t] + mx[pb][i];
      if (t < T) a.y[(size_t)(b * T + t) * H * P + (size_t)h * P + p] = acc;
    }
  }
}

template <int N>
hipError_t launch_n(const ScanArgs& a, hipStream_t s) {
  const bool multi = a.S_final != nullptr || a.T > a.chunk;
  constexpr int lds_multi = ScanLds<N>::BYTES;
  if (multi) {
    auto kern = ssd_scan_kernel<N>;
    hipLaunchKernelGGL(kern, dim3(a.B * a.H), dim3(64), lds_multi, s, a);
  } else {
    // heads in groups of SCAN_HW that share B and C: one workgroup per group of heads
    const bool grouped = a.S0_h16 && a.H % SCAN_HW == 0 && (a.H / a.G) % SCAN_HW == 0;
    if (grouped) hipLaunchKernelGGL(ssd_scan_grp<N>, dim3(a.B * (a.H / SCAN_HW)), dim3(64 * SCAN_HW), 0, s, a);
    else if (a.S0_h16) hipLaunchKernelGGL((ssd_scan_one<N, true>), dim3(a.B * a.H), dim3(64), 0, s, a);
    else hipLaunchKernelGGL((ssd_scan_one<N, false>), dim3(a.B * a.H), dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ssd_scan(const ScanArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.T <= 0 || a.H <= 0) return hipSuccess;
  if (a.P != P || a.chunk < 1 || a.chunk > QMAX) return hipErrorInvalidValue;
  switch (a.N) {
    case 16: return launch_n<16>(a, s);
    case 32: return launch_n<32>(a, s);
    case 64: return launch_n<64>(a, s);
    case 128: return launch_n<128>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hspec
