// bf16 MFMA GEMM for the drafting step's projections:  C[M,N] = A[M,K] * W[N,K]^T (+ R).
//
// Both operands are K-contiguous (PyTorch Linear layout W[out, in]).  An operand may carry
// a second bf16 plane holding the rounding residual of an fp32 value (x = hi + lo); the
// products hi*hi + lo*hi + hi*lo then reproduce fp32 operands to ~2^-16 relative.
//
// Tiling: 4 waves per workgroup in a WM x WN grid, each wave owns TM x TN blocks of 32x32
// computed with v_mfma_f32_32x32x16_bf16.  K is consumed in 64-wide tiles staged through
// LDS (16-byte chunks, XOR-swizzled by row so the per-lane fragment reads of 32 rows spread
// over all banks); the next tile's global loads are issued before the current tile is
// multiplied.  Workgroup ids are remapped so that consecutive output tiles that share a
// weight tile land on the same XCD (its own L2), and every weight byte is fetched from
// HBM once.
#include "common.h"
#include "kernels.h"

namespace hspec {

namespace {

constexpr int BK = 64;          // k-tile (elements); 128 bytes per row
constexpr int CPR = BK / 8;     // 16-byte chunks per row

template <int WM, int WN, int TM, int TN, bool ALO, bool WLO>
struct GemmCfg {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int BM = WM * TM * 32;
  static constexpr int BN = WN * TN * 32;
  static constexpr int A_CH = BM * CPR / NT;   // A chunks per thread per plane
  static constexpr int W_CH = BN * CPR / NT;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile/threads mismatch");
  static constexpr int LDS_A = BM * BK;        // elements per plane
  static constexpr int LDS_W = BN * BK;
  static constexpr int LDS_BYTES = 2 * (LDS_A * (ALO ? 2 : 1) + LDS_W * (WLO ? 2 : 1));
};

__device__ __forceinline__ int swz(int row, int chunk) { return row * CPR + (chunk ^ (row & 7)); }

__device__ __forceinline__ bf16x8 ld_chunk(const bf16* base, int ld, int row, int col, int rows, int K) {
  if (row < rows && col < K) return ld8(base + (size_t)row * ld + col);
  return zero8();
}

// Map a linear workgroup id to a (m-tile, n-tile) pair: ids on the same XCD (id % 8) get
// consecutive virtual ids, and consecutive virtual ids walk the m-tiles of one n-tile.
__device__ __forceinline__ void tile_of(int id, int total, int mt_count, int& mt, int& nt) {
  int per = total / 8, rem = total % 8;
  int x = id % 8, j = id / 8;
  int v = x * per + (x < rem ? x : rem) + j;
  mt = v % mt_count;
  nt = v / mt_count;
}

template <int WM, int WN, int TM, int TN, bool ALO, bool WLO>
__global__ void __launch_bounds__(64 * WM * WN)
gemm_kernel(GemmArgs g) {
  using C = GemmCfg<WM, WN, TM, TN, ALO, WLO>;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* sA = reinterpret_cast<bf16*>(smem);
  bf16* sAl = sA + C::LDS_A;
  bf16* sW = sA + C::LDS_A * (ALO ? 2 : 1);
  bf16* sWl = sW + C::LDS_W;

  const int mt_count = (g.M + C::BM - 1) / C::BM;
  const int nt_count = (g.N + C::BN - 1) / C::BN;
  int mt, nt;
  tile_of(blockIdx.x, mt_count * nt_count, mt_count, mt, nt);
  const int m0 = mt * C::BM, n0 = nt * C::BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  bf16x8 ra[C::A_CH], ral[ALO ? C::A_CH : 1], rw[C::W_CH], rwl[WLO ? C::W_CH : 1];

  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
      int q = i * C::NT + tid, r = q / CPR, c = q % CPR;
      ra[i] = ld_chunk(g.A_hi + (size_t)m0 * g.lda, g.lda, r, k0 + 8 * c, g.M - m0, g.K);
      if constexpr (ALO) ral[i] = ld_chunk(g.A_lo + (size_t)m0 * g.lda, g.lda, r, k0 + 8 * c, g.M - m0, g.K);
    }
#pragma unroll
    for (int i = 0; i < C::W_CH; ++i) {
      int q = i * C::NT + tid, r = q / CPR, c = q % CPR;
      rw[i] = ld_chunk(g.W_hi + (size_t)n0 * g.ldw, g.ldw, r, k0 + 8 * c, g.N - n0, g.K);
      if constexpr (WLO) rwl[i] = ld_chunk(g.W_lo + (size_t)n0 * g.ldw, g.ldw, r, k0 + 8 * c, g.N - n0, g.K);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
      int q = i * C::NT + tid, r = q / CPR, c = q % CPR;
      *reinterpret_cast<bf16x8*>(sA + 8 * swz(r, c)) = ra[i];
      if constexpr (ALO) *reinterpret_cast<bf16x8*>(sAl + 8 * swz(r, c)) = ral[i];
    }
#pragma unroll
    for (int i = 0; i < C::W_CH; ++i) {
      int q = i * C::NT + tid, r = q / CPR, c = q % CPR;
      *reinterpret_cast<bf16x8*>(sW + 8 * swz(r, c)) = rw[i];
      if constexpr (WLO) *reinterpret_cast<bf16x8*>(sWl + 8 * swz(r, c)) = rwl[i];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  const int nk = (g.K + BK - 1) / BK;
  load(0);
  for (int kt = 0; kt < nk; ++kt) {
    __syncthreads();
    store();
    __syncthreads();
    if (kt + 1 < nk) load((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = 2 * ks + (lane >> 5);
      bf16x8 fa[TM], fal[ALO ? TM : 1], fw[TN], fwl[WLO ? TN : 1];
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        int r = (wm * TM + a) * 32 + (lane & 31);
        fa[a] = *reinterpret_cast<const bf16x8*>(sA + 8 * swz(r, ch));
        if constexpr (ALO) fal[a] = *reinterpret_cast<const bf16x8*>(sAl + 8 * swz(r, ch));
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        int r = (wn * TN + b) * 32 + (lane & 31);
        fw[b] = *reinterpret_cast<const bf16x8*>(sW + 8 * swz(r, ch));
        if constexpr (WLO) fwl[b] = *reinterpret_cast<const bf16x8*>(sWl + 8 * swz(r, ch));
      }
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          acc[a][b] = mma32(fa[a], fw[b], acc[a][b]);
          if constexpr (ALO) acc[a][b] = mma32(fal[a], fw[b], acc[a][b]);
          if constexpr (WLO) acc[a][b] = mma32(fa[a], fwl[b], acc[a][b]);
        }
    }
  }

  // Epilogue: lane holds rows 8(i/4)+4(l/32)+i%4 of column l%32 of each 32x32 block.
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int n = n0 + (wn * TN + b) * 32 + (lane & 31);
      if (n >= g.N) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = m0 + (wm * TM + a) * 32 + 8 * (i / 4) + 4 * (lane >> 5) + (i % 4);
        if (m >= g.M) continue;
        float v = acc[a][b][i];
        if (g.R) {
          v += g.r_bf16 ? bf2f(reinterpret_cast<const bf16*>(g.R)[(size_t)m * g.ldr + n])
                        : reinterpret_cast<const float*>(g.R)[(size_t)m * g.ldr + n];
        }
        if (g.C) g.C[(size_t)m * g.ldc + n] = v;
        if (g.C_hi) {
          bf16 h = f2bf(v);
          g.C_hi[(size_t)m * g.ldch + n] = h;
          if (g.C_lo) g.C_lo[(size_t)m * g.ldch + n] = f2bf(v - bf2f(h));
        }
      }
    }
}

template <int WM, int WN, int TM, int TN, bool ALO, bool WLO>
hipError_t launch_one(const GemmArgs& g, hipStream_t s) {
  using C = GemmCfg<WM, WN, TM, TN, ALO, WLO>;
  auto kern = gemm_kernel<WM, WN, TM, TN, ALO, WLO>;
  const int tiles = ((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  if (C::LDS_BYTES > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(C::NT), C::LDS_BYTES, s, g);
  return hipGetLastError();
}

template <int WM, int WN, int TM, int TN>
hipError_t launch_cfg(const GemmArgs& g, hipStream_t s) {
  const bool alo = g.A_lo != nullptr, wlo = g.W_lo != nullptr;
  if (!alo && !wlo) return launch_one<WM, WN, TM, TN, false, false>(g, s);
  if (alo && !wlo) return launch_one<WM, WN, TM, TN, true, false>(g, s);
  if (!alo && wlo) return launch_one<WM, WN, TM, TN, false, true>(g, s);
  return launch_one<WM, WN, TM, TN, true, true>(g, s);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.M <= 64) return launch_cfg<1, 4, 2, 2>(g, s);      // 64 x 256: weight streaming
  if (g.M <= 128) return launch_cfg<2, 2, 2, 4>(g, s);     // 128 x 256
  return launch_cfg<2, 2, 2, 2>(g, s);                     // 128 x 128: dense
}

}  // namespace hspec
