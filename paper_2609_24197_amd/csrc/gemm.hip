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
//
// Few rows (M <= 64, e.g. the state projection of one step's B requests) make the product a
// stream over W: each weight byte feeds at most 64 rows, far below the MFMA/HBM balance
// point, so that path skips LDS for W.  Every lane loads its 16-byte B fragment of
// v_mfma_f32_16x16x32_bf16 straight from HBM (buffer loads whose range check zero-fills rows
// past N), several k-steps ahead, while the small A operand is staged once per workgroup in
// LDS and shared by its waves.  Narrow N is split over K with a fixed-order reduction.
// A weight read this way touches each 128-byte line in two halves a k-step apart, which caps
// HBM efficiency; the packed layout (launch_pack_w) stores every 16x32 operand fragment as
// one contiguous 1 KB block, k-step-major, so that the whole grid sweeps W in address order
// with non-temporal loads.
#include <utility>

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

// ---------------------------------------------------------------- weight-streaming path

constexpr int SK_KC = 128;                  // k per LDS chunk of A
constexpr int SK_STEP = 32;                 // k per MFMA (16x16x32)
constexpr int SK_SPC = SK_KC / SK_STEP;     // k-steps per chunk; also the W prefetch depth
constexpr int SK_OOB = 0x7fffff00;          // buffer offset beyond every range: reads zeros

template <int MT, int NTW, int NW, bool ALO>
struct SkCfg {
  static constexpr int NT = 64 * NW;
  static constexpr int BN = NW * NTW * 16;            // columns per workgroup
  static constexpr int ROWS = MT * 16;
  static constexpr int PLANE = ROWS * SK_KC;          // elements of one A plane per stage
  static constexpr int STAGE = PLANE * (ALO ? 2 : 1);
  static constexpr int CHUNKS = STAGE / 8;            // 16-byte pieces per stage
  static constexpr int A_PT = (CHUNKS + NT - 1) / NT;
};

__device__ __forceinline__ void lds_barrier() {
  // ds_write completion (lgkmcnt 0, vmcnt/expcnt untouched), then the workgroup barrier
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// C[M, N] (or split-K partials) for M <= 16 * MT.  Workgroup = (column tile, k-part); wave w
// owns NTW 16-column tiles and all rows.  A chunk (k0, k0 + 128) of every A plane sits in LDS
// with the 16-byte piece c of row m at c ^ (m & 15), so the fragment reads of 16 rows hit
// distinct banks.
template <int MT, int NTW, int NW, bool ALO, bool PK>
__global__ void __launch_bounds__(64 * NW)
skinny_kernel(GemmArgs g, int kper) {
  using S = SkCfg<MT, NTW, NW, ALO>;
  __shared__ __align__(16) bf16 sA[2 * S::STAGE];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntiles = (g.N + S::BN - 1) / S::BN;
  const int tile = blockIdx.x % ntiles, kp = blockIdx.x / ntiles;
  const int kb = kp * kper, ke = min(g.K, kb + kper);
  const int nsteps = (ke - kb) / SK_STEP;
  const int nch = (ke - kb + SK_KC - 1) / SK_KC;
  const int n_w = tile * S::BN + wave * NTW * 16;

  // W: lane l needs row n_w + 16 j + l % 16 at k offset 8 (l / 16) of each k-step.
  // Row-major: one buffer resource over the wave's rows (rows past N read as zeros).
  // Packed: per k-step, the wave's NTW tiles are one contiguous range of 1 KB fragments.
  const int rows_w = max(0, min(NTW * 16, g.N - n_w));
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(g.W_hi + (size_t)min(n_w, g.N) * g.ldw), 0, __builtin_amdgcn_readfirstlane(rows_w * g.ldw * 2),
      0x00020000);
  int voff[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
    voff[j] = PK ? j * 1024 + lane * 16 : ((16 * j + (lane & 15)) * g.ldw + kb + 8 * (lane >> 4)) * 2;
  const int ntile = g.N / 16, t0 = min(n_w / 16, ntile);
  const int tiles_w = min(NTW, ntile - t0);

  bf16x8 wr[SK_SPC][NTW];
  auto load_w = [&](int st, bf16x8 (&slot)[NTW]) {
    if constexpr (PK) {
      const bool live = st < nsteps;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(g.W_hi + ((size_t)(kb / SK_STEP + (live ? st : 0)) * ntile + t0) * 512), 0,
          __builtin_amdgcn_readfirstlane(live ? tiles_w * 1024 : 0), 0x00020000);
#pragma unroll
      for (int j = 0; j < NTW; ++j)   // aux 2: non-temporal, W is read once
        slot[j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, voff[j], 0, 2));
    } else {
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int off = st < nsteps ? voff[j] + st * SK_STEP * 2 : SK_OOB;
        slot[j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0));
      }
    }
  };

  // A: buffer resources over the M rows of each plane (rows past M and pieces past ke read
  // as zeros), so every load below is unconditional and the wait counts stay exact.
  const __amdgpu_buffer_rsrc_t ra_hi = __builtin_amdgcn_make_buffer_rsrc(
      (void*)g.A_hi, 0, __builtin_amdgcn_readfirstlane(g.M * g.lda * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t ra_lo = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(ALO ? g.A_lo : g.A_hi), 0, __builtin_amdgcn_readfirstlane(g.M * g.lda * 2), 0x00020000);
  bf16x8 ar[S::A_PT];
  auto load_a = [&](int c) {
    const int k0 = kb + c * SK_KC;
#pragma unroll
    for (int i = 0; i < S::A_PT; ++i) {
      const int q = tid + i * S::NT;
      if (S::CHUNKS % S::NT != 0 && q >= S::CHUNKS) continue;
      const int plane = q / (S::ROWS * 16), rem = q % (S::ROWS * 16), m = rem / 16, cc = rem % 16;
      const int k = k0 + 8 * cc;
      const int off = (c < nch && k < ke) ? (m * g.lda + k) * 2 : SK_OOB;
      if constexpr ((S::ROWS * 16) % S::NT == 0) {
        // the plane of piece i is the same in every lane
        const bool lo = (i * S::NT) / (S::ROWS * 16) != 0;
        ar[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(lo ? ra_lo : ra_hi, off, 0, 0));
      } else {
        // lanes of both planes: each lane reads its own piece; the other load reads zeros
        const u32x4 h = __builtin_amdgcn_raw_buffer_load_b128(ra_hi, plane ? SK_OOB : off, 0, 0);
        const u32x4 l = __builtin_amdgcn_raw_buffer_load_b128(ra_lo, plane ? off : SK_OOB, 0, 0);
        ar[i] = __builtin_bit_cast(bf16x8, h | l);
      }
    }
  };
  auto store_a = [&](int stage) {
    bf16* dst = sA + stage * S::STAGE;
#pragma unroll
    for (int i = 0; i < S::A_PT; ++i) {
      const int q = tid + i * S::NT;
      if (S::CHUNKS % S::NT != 0 && q >= S::CHUNKS) continue;
      const int plane = q / (S::ROWS * 16), rem = q % (S::ROWS * 16), m = rem / 16, cc = rem % 16;
      *reinterpret_cast<bf16x8*>(dst + plane * S::PLANE + m * SK_KC + 8 * (cc ^ (m & 15))) = ar[i];
    }
  };

  f32x4 acc[MT][NTW];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[t][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_a(0);
#pragma unroll
  for (int p = 0; p < SK_SPC; ++p) load_w(p, wr[p]);
  store_a(0);
  lds_barrier();
  for (int c = 0; c < nch; ++c) {
    const bf16* sa = sA + (c & 1) * S::STAGE;
    load_a(c + 1);
#pragma unroll
    for (int ks = 0; ks < SK_SPC; ++ks) {
      bf16x8 fa[MT], fl[ALO ? MT : 1];
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int m = 16 * t + (lane & 15), cc = 4 * ks + (lane >> 4);
        const bf16* p = sa + m * SK_KC + 8 * (cc ^ (m & 15));
        fa[t] = *reinterpret_cast<const bf16x8*>(p);
        if constexpr (ALO) fl[t] = *reinterpret_cast<const bf16x8*>(p + S::PLANE);
      }
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          acc[t][j] = mma16(fa[t], wr[ks][j], acc[t][j]);
          if constexpr (ALO) acc[t][j] = mma16(fl[t], wr[ks][j], acc[t][j]);
        }
      load_w((c + 1) * SK_SPC + ks, wr[ks]);
      __builtin_amdgcn_sched_barrier(0);   // keep each step's refill behind its own MFMAs
    }
    store_a((c + 1) & 1);
    lds_barrier();
  }

  // lane holds rows 16 t + 4 (l / 16) + i of column 16 j + l % 16
  const bool split = gridDim.x > ntiles;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int n = n_w + 16 * j + (lane & 15);
      if (n >= g.N) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 16 * t + 4 * (lane >> 4) + i;
        if (m >= g.M) continue;
        float v = acc[t][j][i];
        if (split) {
          g.part[((size_t)kp * g.M + m) * g.N + n] = v;
          continue;
        }
        if (g.R) {
          v += g.r_bf16 ? bf2f(reinterpret_cast<const bf16*>(g.R)[(size_t)m * g.ldr + n])
                        : reinterpret_cast<const float*>(g.R)[(size_t)m * g.ldr + n];
        }
        if (g.C) g.C[(size_t)m * g.ldc + n] = v;
        if (g.C_hi) {
          const bf16 h = f2bf(v);
          g.C_hi[(size_t)m * g.ldch + n] = h;
          if (g.C_lo) g.C_lo[(size_t)m * g.ldch + n] = f2bf(v - bf2f(h));
        }
      }
    }
}

// Sum of the split-K partials in k-part order, then the usual epilogue.
__global__ void __launch_bounds__(256) skinny_reduce(GemmArgs g, int nparts) {
  const size_t total = (size_t)g.M * g.N;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
    const int m = (int)(e / g.N), n = (int)(e % g.N);
    float v = 0.f;
    for (int p = 0; p < nparts; ++p) v += g.part[(size_t)p * total + e];
    if (g.R) {
      v += g.r_bf16 ? bf2f(reinterpret_cast<const bf16*>(g.R)[(size_t)m * g.ldr + n])
                    : reinterpret_cast<const float*>(g.R)[(size_t)m * g.ldr + n];
    }
    if (g.C) g.C[(size_t)m * g.ldc + n] = v;
    if (g.C_hi) {
      const bf16 h = f2bf(v);
      g.C_hi[(size_t)m * g.ldch + n] = h;
      if (g.C_lo) g.C_lo[(size_t)m * g.ldch + n] = f2bf(v - bf2f(h));
    }
  }
}

int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cus[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

constexpr int SK_NW = 8;

// Launch shape of the weight-streaming path: wide N uses 4 column tiles per wave; narrow N
// uses 1 and splits K until the grid covers the chip twice.
struct SkPlan {
  bool use = false;
  int ntw = 4, ksplit = 1, kper = 0;
};

SkPlan skinny_plan(int M, int N, int K, bool w_lo, int cus) {
  SkPlan p;
  if (M > 64 || w_lo || K % SK_STEP != 0) return p;
  p.use = true;
  const int want = 2 * cus;
  int tiles = (N + SK_NW * 64 - 1) / (SK_NW * 64);
  if (tiles < want) {
    p.ntw = 1;
    tiles = (N + SK_NW * 16 - 1) / (SK_NW * 16);
  }
  const int kch = (K + SK_KC - 1) / SK_KC;
  int ks = tiles >= want ? 1 : (want + tiles - 1) / tiles;
  if (ks > kch) ks = kch;
  if (ks < 1) ks = 1;
  p.kper = ((kch + ks - 1) / ks) * SK_KC;
  p.ksplit = (K + p.kper - 1) / p.kper;
  return p;
}

template <int MT, int NTW, bool ALO, bool PK>
hipError_t launch_skinny_t(const GemmArgs& g, const SkPlan& p, hipStream_t s) {
  using S = SkCfg<MT, NTW, SK_NW, ALO>;
  auto kern = skinny_kernel<MT, NTW, SK_NW, ALO, PK>;
  const int ntiles = (g.N + S::BN - 1) / S::BN;
  hipLaunchKernelGGL(kern, dim3(ntiles * p.ksplit), dim3(S::NT), 0, s, g, p.kper);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.ksplit == 1) return e;
  const size_t total = (size_t)g.M * g.N;
  size_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(skinny_reduce, dim3((unsigned)blocks), dim3(256), 0, s, g, p.ksplit);
  return hipGetLastError();
}

template <int MT, bool ALO>
hipError_t launch_skinny_m(const GemmArgs& g, const SkPlan& p, hipStream_t s) {
  if (g.w_packed) return p.ntw == 4 ? launch_skinny_t<MT, 4, ALO, true>(g, p, s) : launch_skinny_t<MT, 1, ALO, true>(g, p, s);
  return p.ntw == 4 ? launch_skinny_t<MT, 4, ALO, false>(g, p, s) : launch_skinny_t<MT, 1, ALO, false>(g, p, s);
}

template <bool ALO>
hipError_t launch_skinny_a(const GemmArgs& g, const SkPlan& p, hipStream_t s) {
  if (g.M <= 16) return launch_skinny_m<1, ALO>(g, p, s);
  if (g.M <= 32) return launch_skinny_m<2, ALO>(g, p, s);
  return launch_skinny_m<4, ALO>(g, p, s);
}

// ------------------------------------------------------------- pipelined dense path
//
// Many rows (M >= 128): 128 x 128 output tiles, 4 waves of 64 x 64 (v_mfma_f32_32x32x16_bf16).
// A and W k-tiles (64 wide) go straight from global memory into LDS (global_load_lds_dwordx4),
// ST stages deep, so ST-1 tiles are in flight while one is multiplied; every LDS stage is its
// own object so that the compiler's wait for outstanding LDS DMA names only the stage being
// read.  Rows past M or N re-read the last valid row (their results are never stored); K must
// be a multiple of 64.

template <int TM, int TN, bool ALO, int ST>
struct DmaCfg {
  static constexpr int NT = 256;
  static constexpr int BM = 2 * TM * 32, BN = 2 * TN * 32;
  static constexpr int SA = BM * BK, SW = BN * BK;                  // elements per plane per stage
  static constexpr int STAGE = SA * (ALO ? 2 : 1) + SW;
  static constexpr int A_I = BM * CPR / NT, W_I = BN * CPR / NT;   // DMA instructions per wave
  static constexpr int NI = A_I * (ALO ? 2 : 1) + W_I;
  static constexpr int VM = (ST - 2) * NI;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0 && VM < 64 && ST >= 2 && ST <= 4, "dma gemm shape");
};

__device__ __forceinline__ void dma16(const bf16* src, bf16* lds) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
  // vmcnt <= VM and every LDS read of this wave complete
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (0 << 8) | ((VM >> 4) << 14));
  asm volatile("" ::: "memory");
}

// Epilogue of a 32x32 accumulator block: lane holds rows 8(i/4)+4(l/32)+i%4 of column l%32.
__device__ __forceinline__ void store_block32(const GemmArgs& g, const f32x16& acc, int mb, int nb, int lane) {
  const int n = nb + (lane & 31);
  if (n >= g.N) return;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int m = mb + 8 * (i / 4) + 4 * (lane >> 5) + (i % 4);
    if (m >= g.M) continue;
    float v = acc[i];
    if (g.R) {
      v += g.r_bf16 ? bf2f(reinterpret_cast<const bf16*>(g.R)[(size_t)m * g.ldr + n])
                    : reinterpret_cast<const float*>(g.R)[(size_t)m * g.ldr + n];
    }
    if (g.C) g.C[(size_t)m * g.ldc + n] = v;
    if (g.C_hi) {
      const bf16 h = f2bf(v);
      g.C_hi[(size_t)m * g.ldch + n] = h;
      if (g.C_lo) g.C_lo[(size_t)m * g.ldch + n] = f2bf(v - bf2f(h));
    }
  }
}

template <int TM, int TN, bool ALO, int ST>
__global__ void __launch_bounds__(256) gemm_dma_kernel(GemmArgs g) {
  using C = DmaCfg<TM, TN, ALO, ST>;
  // one LDS object per (stage, operand): the A planes and the W tile of stage s
  constexpr int PA = C::SA * (ALO ? 2 : 1);
  __shared__ __align__(16) bf16 A0s[PA], W0s[C::SW];
  __shared__ __align__(16) bf16 A1s[PA], W1s[C::SW];
  __shared__ __align__(16) bf16 A2s[ST > 2 ? PA : 8], W2s[ST > 2 ? C::SW : 8];
  __shared__ __align__(16) bf16 A3s[ST > 3 ? PA : 8], W3s[ST > 3 ? C::SW : 8];
  auto sa_of = [&](auto I) -> bf16* {
    if constexpr (decltype(I)::value == 0) return A0s;
    else if constexpr (decltype(I)::value == 1) return A1s;
    else if constexpr (decltype(I)::value == 2) return A2s;
    else return A3s;
  };
  auto sw_of = [&](auto I) -> bf16* {
    if constexpr (decltype(I)::value == 0) return W0s;
    else if constexpr (decltype(I)::value == 1) return W1s;
    else if constexpr (decltype(I)::value == 2) return W2s;
    else return W3s;
  };

  const int mt_count = (g.M + C::BM - 1) / C::BM;
  const int nt_count = (g.N + C::BN - 1) / C::BN;
  int mt, nt;
  tile_of(blockIdx.x, mt_count * nt_count, mt_count, mt, nt);
  const int m0 = mt * C::BM, n0 = nt * C::BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / 2, wn = wave % 2;

  const int rows_a = min(C::BM, g.M - m0), rows_w = min(C::BN, g.N - n0);
  const bf16* A0 = g.A_hi + (size_t)m0 * g.lda;
  const bf16* Al0 = (ALO ? g.A_lo : g.A_hi) + (size_t)m0 * g.lda;
  const bf16* W0 = g.W_hi + (size_t)n0 * g.ldw;

  // unit u (16 bytes) of a stage plane: row u / 8, stored chunk u % 8 = logical chunk ^ (row & 7)
  auto issue = [&](int t, bf16* L, bf16* LW) {
    const int k0 = t * BK;
#pragma unroll
    for (int i = 0; i < C::A_I; ++i) {
      const int u0 = (i * 4 + wave) * 64, u = u0 + lane, row = u >> 3, k = k0 + 8 * ((u & 7) ^ (row & 7));
      const size_t off = (size_t)min(row, rows_a - 1) * g.lda + k;
      dma16(A0 + off, L + u0 * 8);
      if constexpr (ALO) dma16(Al0 + off, L + C::SA + u0 * 8);
    }
#pragma unroll
    for (int i = 0; i < C::W_I; ++i) {
      const int u0 = (i * 4 + wave) * 64, u = u0 + lane, row = u >> 3, k = k0 + 8 * ((u & 7) ^ (row & 7));
      dma16(W0 + (size_t)min(row, rows_w - 1) * g.ldw + k, LW + u0 * 8);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  auto compute = [&](const bf16* L, const bf16* LW) {
    const bf16* sA = L;
    const bf16* sAl = L + C::SA;
    const bf16* sW = LW;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = 2 * ks + (lane >> 5);
      bf16x8 fa[TM], fal[ALO ? TM : 1], fw[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const int r = (wm * TM + a) * 32 + (lane & 31);
        fa[a] = *reinterpret_cast<const bf16x8*>(sA + 8 * swz(r, ch));
        if constexpr (ALO) fal[a] = *reinterpret_cast<const bf16x8*>(sAl + 8 * swz(r, ch));
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int r = (wn * TN + b) * 32 + (lane & 31);
        fw[b] = *reinterpret_cast<const bf16x8*>(sW + 8 * swz(r, ch));
      }
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          acc[a][b] = mma32(fa[a], fw[b], acc[a][b]);
          if constexpr (ALO) acc[a][b] = mma32(fal[a], fw[b], acc[a][b]);
        }
    }
  };

  const int nk = (g.K + BK - 1) / BK;
  // prologue without branches (tiles past the end re-read the last one into unused stages),
  // so that the compiler's record of which stage each pending DMA fills stays exact
  [&]<int... I>(std::integer_sequence<int, I...>) {
    (issue(min(I, nk - 1), sa_of(Int<I>{}), sw_of(Int<I>{})), ...);
  }(std::make_integer_sequence<int, ST - 1>{});
  // steady state: straight-line rounds of ST steps, each waiting for its own tile only
  auto steady = [&](int t, auto S) {
    wait_vm_lgkm0<C::VM>();
    wg_barrier();   // tile t is in LDS for every wave; every wave is done reading tile t-1
    constexpr int N = (decltype(S)::value + ST - 1) % ST;
    issue(t + ST - 1, sa_of(Int<N>{}), sw_of(Int<N>{}));
    compute(sa_of(S), sw_of(S));
  };
  auto step = [&](int t, auto S) {
    if (t + ST - 2 < nk) wait_vm_lgkm0<C::VM>();
    else wait_vm_lgkm0<0>();
    wg_barrier();
    constexpr int N = (decltype(S)::value + ST - 1) % ST;
    if (t + ST - 1 < nk) issue(t + ST - 1, sa_of(Int<N>{}), sw_of(Int<N>{}));
    compute(sa_of(S), sw_of(S));
  };
  int t0 = 0;
  for (; t0 + 2 * ST - 2 < nk; t0 += ST) {
    [&]<int... I>(std::integer_sequence<int, I...>) {
      (steady(t0 + I, Int<I>{}), ...);
    }(std::make_integer_sequence<int, ST>{});
  }
  for (; t0 < nk; t0 += ST) {
    [&]<int... I>(std::integer_sequence<int, I...>) {
      ((t0 + I < nk ? step(t0 + I, Int<I>{}) : void()), ...);
    }(std::make_integer_sequence<int, ST>{});
  }

#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
      store_block32(g, acc[a][b], m0 + (wm * TM + a) * 32, n0 + (wn * TN + b) * 32, lane);
}

template <int TM, int TN, bool ALO, int ST>
hipError_t launch_dma(const GemmArgs& g, hipStream_t s) {
  using C = DmaCfg<TM, TN, ALO, ST>;
  const int tiles = ((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_dma_kernel<TM, TN, ALO, ST>), dim3(tiles), dim3(C::NT), 0, s, g);
  return hipGetLastError();
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

__global__ void __launch_bounds__(256) pack_w_kernel(const bf16* __restrict__ W, int N, int K, bf16* __restrict__ Wp) {
  // one 16-byte piece (row n, columns 8q..8q+7) per thread and iteration
  const int qr = K / 8, ntile = N / 16;
  const size_t total = (size_t)N * qr;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
    const int n = (int)(e / qr), q = (int)(e % qr);
    const int st = q / 4, c = q % 4, t = n / 16, i = n % 16;
    const size_t dst = (((size_t)st * ntile + t) * 64 + i + 16 * c) * 8;
    *reinterpret_cast<bf16x8*>(Wp + dst) = ld8(W + (size_t)n * K + 8 * q);
  }
}

}  // namespace

hipError_t launch_pack_w(const bf16* W, int N, int K, bf16* Wp, hipStream_t s) {
  if (N % 16 || K % SK_STEP || N <= 0 || K <= 0) return hipErrorInvalidValue;
  const size_t total = (size_t)N * (K / 8);
  size_t blocks = (total + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W, N, K, Wp);
  return hipGetLastError();
}

size_t gemm_scratch_elems(int M, int N, int K, bool a_lo, bool w_lo) {
  (void)a_lo;
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  const SkPlan p = skinny_plan(M, N, K, w_lo, device_cus());
  return p.use && p.ksplit > 1 ? (size_t)p.ksplit * M * N : 0;
}

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  SkPlan p = skinny_plan(g.M, g.N, g.K, g.W_lo != nullptr, device_cus());
  if (g.w_packed && (!p.use || g.N % 16 || g.W_lo)) return hipErrorInvalidValue;   // packed W needs this path
  if (p.use) {
    if (p.ksplit > 1 && (!g.part || g.part_cap < (size_t)p.ksplit * g.M * g.N)) {
      p.ksplit = 1;
      p.kper = ((g.K + SK_KC - 1) / SK_KC) * SK_KC;
    }
    return g.A_lo ? launch_skinny_a<true>(g, p, s) : launch_skinny_a<false>(g, p, s);
  }
  if (g.M <= 64) return launch_cfg<1, 4, 2, 2>(g, s);      // 64 x 256: weight streaming
  if (!g.W_lo && g.K % BK == 0)
    return g.A_lo ? launch_dma<2, 2, true, 3>(g, s) : launch_dma<2, 2, false, 4>(g, s);
  if (g.M <= 128) return launch_cfg<2, 2, 2, 4>(g, s);     // 128 x 256
  return launch_cfg<2, 2, 2, 2>(g, s);                     // 128 x 128: dense
}

}  // namespace hspec
