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
// one contiguous 1 KB block, and the blocks of 32 consecutive 16-row tiles (512 rows, one
// workgroup's item at 64 rows) k-step after k-step, so that each workgroup streams one
// contiguous 4 MB run per item with non-temporal loads (measured against k-step-major blocks,
// where a workgroup reads 32 KB runs 64 MB apart: state projection 1428 -> 1407 us at
// 8b-serving-b64, bitwise the same result).  The packed W holds fp16 values (scaled by a power of two so that
// every bf16 weight converts exactly) and is multiplied with fp16 A planes by
// v_mfma_f32_16x16x32_f16: one fp16 plane of an activation carries 11 significant bits where
// a bf16 plane carries 8, so one product does what a bf16 hi/lo pair would otherwise be needed
// for.  More than 128 rows run as 128-row launches, one after the other.
#include <algorithm>
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

// LDS position (16-byte units) of chunk `chunk` of tile row `row`: the chunk is XOR-ed with
// (row / 2) % 8 so that the 16 rows one ds_read_b128 pass serves (two per 256-byte bank line)
// fall on 16 distinct 4-bank groups.
__device__ __forceinline__ int swz_key(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swz(int row, int chunk) { return row * CPR + (chunk ^ swz_key(row)); }

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

#ifndef HSPEC_SK_KC
#define HSPEC_SK_KC 128
#endif
#ifndef HSPEC_SK_P
#define HSPEC_SK_P 4
#endif
#ifndef HSPEC_SK_NW
#define HSPEC_SK_NW 8
#endif
constexpr int SK_KC = HSPEC_SK_KC;          // k per LDS chunk of A
constexpr int SK_STEP = 32;                 // k per MFMA (16x16x32)
constexpr int SK_SPC = SK_KC / SK_STEP;     // k-steps per chunk
constexpr int SK_CPR = SK_KC / 8;           // 16-byte pieces per row of an A chunk
constexpr int SK_P = HSPEC_SK_P;            // W prefetch depth (k-steps in flight per wave)
static_assert(SK_SPC % SK_P == 0, "prefetch depth must divide the chunk");
constexpr int SK_OOB = 0x7fffff00;          // buffer offset beyond every range: reads zeros
typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));

template <int MT, int NTW, int NW, bool ALO>
struct SkCfg {
  static constexpr int NT = 64 * NW;
  static constexpr int BN = NW * NTW * 16;            // columns per workgroup
  static constexpr int ROWS = MT * 16;
  static constexpr int PLANE = ROWS * SK_KC;          // elements of one A plane per stage
  static constexpr int STAGE = PLANE * (ALO ? 2 : 1);
  static constexpr int CHUNKS = STAGE / 8;            // 16-byte pieces per stage
  static constexpr int A_PT = (CHUNKS + NT - 1) / NT;
  static constexpr int BNW = NTW * 16;                // columns per wave
  static constexpr int PITCH = BNW + 4;               // fp32 row pitch of the epilogue staging
};

__device__ __forceinline__ void lds_barrier() {
  // ds_write completion (lgkmcnt 0, vmcnt/expcnt untouched), then the workgroup barrier
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Buffer resource over [base, base + bytes); a range of 0 bytes makes every access a no-op
// (loads return zeros, stores are dropped).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf(const void* base, long long bytes) {
  const int n = bytes <= 0 ? 0 : (int)(bytes > 0x7fffffffLL ? 0x7fffffff : bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, __builtin_amdgcn_readfirstlane(n), 0x00020000);
}

// Work items are (column tile, k-part) pairs; a workgroup takes items blockIdx.x, +gridDim.x,
// ... so that with a grid of one workgroup per CU the loads of its next tile are already in
// flight while the epilogue of the current one stores.  Wave w owns NTW 16-column tiles and
// all rows of an item.  The A chunk (k0, k0 + SK_KC) of every A plane sits in LDS with the
// 16-byte piece c of row m at c ^ (m & 15), so the fragment reads of 16 rows hit distinct
// banks.  Every global access is an unconditional buffer access whose range check does the
// bounds work, which keeps the compiler's counts of outstanding loads exact across tiles.
template <int MT, int NTW, int NW, bool ALO, bool PK, bool RES>
__global__ void __launch_bounds__(64 * NW)
skinny_kernel(GemmArgs g, int kper, int nitems) {
  using S = SkCfg<MT, NTW, NW, ALO>;
  __shared__ __align__(16) bf16 sA[2 * S::STAGE];
  __shared__ __align__(16) float stg_all[NW * 16 * S::PITCH];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntiles = (g.N + S::BN - 1) / S::BN;
  const int ntile16 = g.N / 16;
  const bool split = nitems > ntiles;

  struct Item {
    int tile, kp, kb, ke, nsteps, nch, n_w;
  };
  auto item_of = [&](int it) {
    Item r;
    r.tile = it % ntiles;
    r.kp = it / ntiles;
    r.kb = r.kp * kper;
    r.ke = min(g.K, r.kb + kper);
    r.nsteps = (r.ke - r.kb) / SK_STEP;
    r.nch = (r.ke - r.kb + SK_KC - 1) / SK_KC;
    r.n_w = r.tile * S::BN + wave * S::BNW;
    return r;
  };

  // ---- W stream: lane l needs row n_w + 16 j + l % 16 at k offset 8 (l / 16) of each k-step
  int vrow[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
    vrow[j] = PK ? j * 1024 + lane * 16 : ((16 * j + (lane & 15)) * g.ldw + 8 * (lane >> 4)) * 2;
  int p_it = blockIdx.x, p_st = 0;          // next k-step to prefetch
  Item p_item = item_of(p_it);
  bf16x8 wr[SK_P][NTW];
  auto load_w_next = [&](bf16x8 (&slot)[NTW]) {
    const bool live = p_it < nitems && p_st < p_item.nsteps;
    if constexpr (PK) {
      // block (k-step s, tile t) of group gr = t / 32 (gs tiles) at gr * 32 * nst + s * gs + t % 32;
      // a wave's NTW tiles share a group (NTW divides 32 and t0 is a multiple of NTW)
      const int t0 = min(p_item.n_w / 16, ntile16);
      const int gr = t0 / 32, gs = min(32, ntile16 - 32 * gr);
      const size_t s_k = (size_t)(p_item.kb / SK_STEP + (live ? p_st : 0));
      const __amdgpu_buffer_rsrc_t rs =
          buf(g.W_hi + ((size_t)gr * 32 * (g.K / SK_STEP) + s_k * gs + (t0 - 32 * gr)) * 512,
              live ? (long long)min(NTW, ntile16 - t0) * 1024 : 0);
#pragma unroll
      for (int j = 0; j < NTW; ++j)   // aux 2: non-temporal, W is read once
        slot[j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, vrow[j], 0, 2));
    } else {
      const int rows = live ? max(0, min(S::BNW, g.N - p_item.n_w)) : 0;
      const __amdgpu_buffer_rsrc_t rs = buf(g.W_hi + (size_t)min(p_item.n_w, g.N) * g.ldw, (long long)rows * g.ldw * 2);
      const int koff = (p_item.kb + p_st * SK_STEP) * 2;
#pragma unroll
      for (int j = 0; j < NTW; ++j)
        slot[j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, vrow[j] + koff, 0, 0));
    }
    if (++p_st == p_item.nch * SK_SPC) {
      p_st = 0;
      p_it += gridDim.x;
      p_item = item_of(p_it);
    }
  };

  // ---- A stream: chunks of the items in order, staged through registers into LDS
  const __amdgpu_buffer_rsrc_t ra_hi = buf(g.A_hi, (long long)g.M * g.lda * 2);
  const __amdgpu_buffer_rsrc_t ra_lo = buf(ALO ? g.A_lo : g.A_hi, (long long)g.M * g.lda * 2);
  int a_it = blockIdx.x, a_c = 0;           // next A chunk to load
  Item a_item = item_of(a_it);
  bf16x8 ar[S::A_PT];
  auto load_a_next = [&]() {
    const bool live = a_it < nitems;
    const int k0 = a_item.kb + a_c * SK_KC;
#pragma unroll
    for (int i = 0; i < S::A_PT; ++i) {
      const int q = tid + i * S::NT;
      if (S::CHUNKS % S::NT != 0 && q >= S::CHUNKS) continue;
      const int plane = q / (S::ROWS * SK_CPR), rem = q % (S::ROWS * SK_CPR), m = rem / SK_CPR, cc = rem % SK_CPR;
      const int k = k0 + 8 * cc;
      const int off = (live && k < a_item.ke) ? (m * g.lda + k) * 2 : SK_OOB;
      if constexpr ((S::ROWS * SK_CPR) % S::NT == 0) {
        // the plane of piece i is the same in every lane
        const bool lo = (i * S::NT) / (S::ROWS * SK_CPR) != 0;
        ar[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(lo ? ra_lo : ra_hi, off, 0, 0));
      } else {
        // lanes of both planes: each lane reads its own piece; the other load reads zeros
        const u32x4 h = __builtin_amdgcn_raw_buffer_load_b128(ra_hi, plane ? SK_OOB : off, 0, 0);
        const u32x4 l = __builtin_amdgcn_raw_buffer_load_b128(ra_lo, plane ? off : SK_OOB, 0, 0);
        ar[i] = __builtin_bit_cast(bf16x8, h | l);
      }
    }
    if (++a_c == a_item.nch) {
      a_c = 0;
      a_it += gridDim.x;
      a_item = item_of(a_it);
    }
  };
  auto store_a = [&](int stage) {
    bf16* dst = sA + stage * S::STAGE;
#pragma unroll
    for (int i = 0; i < S::A_PT; ++i) {
      const int q = tid + i * S::NT;
      if (S::CHUNKS % S::NT != 0 && q >= S::CHUNKS) continue;
      const int plane = q / (S::ROWS * SK_CPR), rem = q % (S::ROWS * SK_CPR), m = rem / SK_CPR, cc = rem % SK_CPR;
      *reinterpret_cast<bf16x8*>(dst + plane * S::PLANE + m * SK_KC + 8 * (cc ^ (m & 15))) = ar[i];
    }
  };

  // ---- epilogue geometry: after staging, lane owns 4 consecutive columns of one row
  float* stg = stg_all + wave * 16 * S::PITCH;
  constexpr int LPR = S::BNW / 4;                    // lanes per row
  constexpr int RPP = 64 / LPR < 16 ? 64 / LPR : 16; // rows per pass
  const int lr = lane / LPR, c4 = (lane % LPR) * 4;

  if (blockIdx.x >= nitems) return;
#pragma unroll
  for (int p = 0; p < SK_P; ++p) load_w_next(wr[p]);
  load_a_next();
  store_a(0);
  lds_barrier();
  int gc = 0;   // chunks consumed by this workgroup: A stage gc & 1

  for (int it = blockIdx.x; it < nitems; it += gridDim.x) {
    const Item cur = item_of(it);
    f32x4 acc[MT][NTW];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int j = 0; j < NTW; ++j) acc[t][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int c = 0; c < cur.nch; ++c, ++gc) {
      const bf16* sa = sA + (gc & 1) * S::STAGE;
      load_a_next();
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
            if constexpr (PK) {   // fp16 operands (the packed layout)
              const f16x8 w16 = __builtin_bit_cast(f16x8, wr[ks % SK_P][j]);
              acc[t][j] = mma16h(__builtin_bit_cast(f16x8, fa[t]), w16, acc[t][j]);
              if constexpr (ALO) acc[t][j] = mma16h(__builtin_bit_cast(f16x8, fl[t]), w16, acc[t][j]);
            } else {
              acc[t][j] = mma16(fa[t], wr[ks % SK_P][j], acc[t][j]);
              if constexpr (ALO) acc[t][j] = mma16(fl[t], wr[ks % SK_P][j], acc[t][j]);
            }
          }
        load_w_next(wr[ks % SK_P]);
        __builtin_amdgcn_sched_barrier(0);   // keep each step's refill behind its own MFMAs
      }
      store_a((gc + 1) & 1);
      lds_barrier();
    }

    // Epilogue (N % 4 == 0): each 16-row slab of the accumulators goes through this wave's LDS
    // staging so that lanes store whole 16-byte pieces of rows.  Outputs outside [0, M) x [0, N)
    // and absent outputs fall outside their buffer's range and are dropped.
    const int n0 = cur.n_w;
    const int cols = max(0, min(S::BNW, g.N - n0));
    const long long rows_span = (long long)(g.M - 1);
    const __amdgpu_buffer_rsrc_t r_part =
        buf(split ? g.part + ((size_t)cur.kp * g.M) * g.N + min(n0, g.N) : nullptr,
            split && cols ? (rows_span * g.N + cols) * 4 : 0);
    const __amdgpu_buffer_rsrc_t r_c =
        buf(g.C ? g.C + min(n0, g.N) : nullptr, !split && g.C && cols ? (rows_span * g.ldc + cols) * 4 : 0);
    const __amdgpu_buffer_rsrc_t r_hi =
        buf(g.C_hi ? g.C_hi + min(n0, g.N) : nullptr, !split && g.C_hi && cols ? (rows_span * g.ldch + cols) * 2 : 0);
    const __amdgpu_buffer_rsrc_t r_lo =
        buf(g.C_lo ? g.C_lo + min(n0, g.N) : nullptr, !split && g.C_lo && cols ? (rows_span * g.ldch + cols) * 2 : 0);
    const __amdgpu_buffer_rsrc_t r_h16 =
        buf(g.C_h16 ? g.C_h16 + min(n0, g.N) : nullptr, !split && g.C_h16 && cols ? (rows_span * g.ldch + cols) * 2 : 0);
    const __amdgpu_buffer_rsrc_t r_l16 =
        buf(g.C_l16 ? g.C_l16 + min(n0, g.N) : nullptr, !split && g.C_l16 && cols ? (rows_span * g.ldch + cols) * 2 : 0);
    const float osc = split ? 1.f : g.out_scale;   // split partials are scaled by the reduction
    // (packed products: exactly one of C_h16 and C, host-checked)
    [[maybe_unused]] const bool h16_only = g.C_h16 != nullptr;
    // residual R (RES: present and not split-K): one of the two loads reads, the other is empty
    const bool rf = RES && !g.r_bf16, rb = RES && g.r_bf16;
    [[maybe_unused]] const __amdgpu_buffer_rsrc_t r_rf =
        buf(rf ? reinterpret_cast<const float*>(g.R) + min(n0, g.N) : nullptr, !split && rf && cols ? (rows_span * g.ldr + cols) * 4 : 0);
    [[maybe_unused]] const __amdgpu_buffer_rsrc_t r_rb =
        buf(rb ? reinterpret_cast<const bf16*>(g.R) + min(n0, g.N) : nullptr, !split && rb && cols ? (rows_span * g.ldr + cols) * 2 : 0);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) stg[(4 * (lane >> 4) + i) * S::PITCH + 16 * j + (lane & 15)] = acc[t][j][i];
      if constexpr (PK) {
        // The packed product writes one output: S0 as one fp16 plane (the step) or fp32 (the
        // state-initialisation entry).  fp16: 8 consecutive columns per lane, one 16-byte store
        // each (against 8-byte stores of 4 columns: 8b-serving-b64 step 2.061 -> 2.023 ms; the
        // output's row layout made no difference).
        if (h16_only) {
          constexpr int L8 = S::BNW / 8, R8 = 64 / L8 < 16 ? 64 / L8 : 16;
          const int lr8 = lane / L8, c8 = (lane % L8) * 8;
#pragma unroll
          for (int pass = 0; pass < 16 / R8; ++pass) {
            const int r = pass * R8 + lr8;
            const int m = 16 * t + r;
            const bool ok = lane < L8 * R8 && m < g.M && c8 < cols;
            const f32x4 v0 = *reinterpret_cast<const f32x4*>(stg + r * S::PITCH + c8) * osc;
            const f32x4 v1 = *reinterpret_cast<const f32x4*>(stg + r * S::PITCH + c8 + 4) * osc;
            f16x8 h8;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              h8[e] = (_Float16)(v0[e] * g.h16_scale);
              h8[4 + e] = (_Float16)(v1[e] * g.h16_scale);
            }
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, h8), r_h16, ok ? (m * g.ldch + c8) * 2 : SK_OOB, 0, 16);
          }
        } else {
#pragma unroll
          for (int pass = 0; pass < 16 / RPP; ++pass) {
            const int r = pass * RPP + lr;
            const int m = 16 * t + r;
            const bool ok = lane < LPR * RPP && m < g.M && c4 < cols;
            const f32x4 v = *reinterpret_cast<const f32x4*>(stg + r * S::PITCH + c4) * osc;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r_c, ok ? (m * g.ldc + c4) * 4 : SK_OOB, 0, 16);
          }
        }
        continue;
      }
#pragma unroll
      for (int pass = 0; pass < 16 / RPP; ++pass) {
        const int r = pass * RPP + lr;
        const int m = 16 * t + r;
        const bool ok = lane < LPR * RPP && m < g.M && c4 < cols;
        f32x4 v = *reinterpret_cast<const f32x4*>(stg + r * S::PITCH + c4) * osc;
        if constexpr (RES) {
          const int o4 = ok ? (m * g.ldr + c4) * 4 : SK_OOB;
          const int o2 = ok ? (m * g.ldr + c4) * 2 : SK_OOB;
          const f32x4 addf = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r_rf, o4, 0, 0));
          const bf16x4 addb = __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r_rb, o2, 0, 0));
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += addf[e] + bf2f(addb[e]);
        }
        bf16x4 h, l;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          h[e] = f2bf(v[e]);
          l[e] = f2bf(v[e] - bf2f(h[e]));
        }
        // aux 16 (sc1): measured to disturb the concurrent non-temporal W stream least
        const u32x4 vb = __builtin_bit_cast(u32x4, v);
        __builtin_amdgcn_raw_buffer_store_b128(vb, r_part, ok ? (m * g.N + c4) * 4 : SK_OOB, 0, 16);
        __builtin_amdgcn_raw_buffer_store_b128(vb, r_c, ok ? (m * g.ldc + c4) * 4 : SK_OOB, 0, 16);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u32, h), r_hi, ok ? (m * g.ldch + c4) * 2 : SK_OOB, 0, 16);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u32, l), r_lo, ok ? (m * g.ldch + c4) * 2 : SK_OOB, 0, 16);
        f16x4 v16, l16;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float sv = v[e] * g.h16_scale;
          v16[e] = (_Float16)sv;
          l16[e] = (_Float16)(sv - (float)v16[e]);
        }
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u32, v16), r_h16, ok ? (m * g.ldch + c4) * 2 : SK_OOB, 0, 16);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u32, l16), r_l16, ok ? (m * g.ldch + c4) * 2 : SK_OOB, 0, 16);
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
    v *= g.out_scale;
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
    if (g.C_h16) {
      const float sv = v * g.h16_scale;
      const _Float16 h = (_Float16)sv;
      g.C_h16[(size_t)m * g.ldch + n] = h;
      if (g.C_l16) g.C_l16[(size_t)m * g.ldch + n] = (_Float16)(sv - (float)h);
    }
  }
}

// The same for 4 consecutive columns per thread (N % 4 == 0, and ldc, ldr, ldch % 4 == 0):
// 16-byte loads of the partials, 8 k-parts issued together, then 16-byte stores.
__global__ void __launch_bounds__(256) skinny_reduce4(GemmArgs g, int nparts) {
  constexpr int GROUP = 8;
  const size_t total = (size_t)g.M * g.N, quads = total / 4;
  for (size_t q = (size_t)blockIdx.x * 256 + threadIdx.x; q < quads; q += (size_t)gridDim.x * 256) {
    const size_t e = q * 4;
    const int m = (int)(e / g.N), n = (int)(e % g.N);
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    for (int p0 = 0; p0 < nparts; p0 += GROUP) {
      f32x4 part[GROUP];
#pragma unroll
      for (int k = 0; k < GROUP; ++k)
        part[k] = p0 + k < nparts ? *reinterpret_cast<const f32x4*>(g.part + (size_t)(p0 + k) * total + e)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < GROUP; ++k) v += part[k];   // absent parts add +0
    }
    v *= g.out_scale;
    if (g.R) {
      if (g.r_bf16) {
        const bf16x4 r = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const bf16*>(g.R) + (size_t)m * g.ldr + n);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] += bf2f(r[i]);
      } else {
        v += *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(g.R) + (size_t)m * g.ldr + n);
      }
    }
    if (g.C) *reinterpret_cast<f32x4*>(g.C + (size_t)m * g.ldc + n) = v;
    if (g.C_hi) {
      bf16x4 h, l;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        h[i] = f2bf(v[i]);
        l[i] = f2bf(v[i] - bf2f(h[i]));
      }
      *reinterpret_cast<bf16x4*>(g.C_hi + (size_t)m * g.ldch + n) = h;
      if (g.C_lo) *reinterpret_cast<bf16x4*>(g.C_lo + (size_t)m * g.ldch + n) = l;
    }
    if (g.C_h16) {
      f16x4 h, l;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sv = v[i] * g.h16_scale;
        h[i] = (_Float16)sv;
        l[i] = (_Float16)(sv - (float)h[i]);
      }
      *reinterpret_cast<f16x4*>(g.C_h16 + (size_t)m * g.ldch + n) = h;
      if (g.C_l16) *reinterpret_cast<f16x4*>(g.C_l16 + (size_t)m * g.ldch + n) = l;
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

constexpr int SK_NW = HSPEC_SK_NW;

// Launch shape of the weight-streaming path: wide N uses 4 column tiles per wave (2 at 65..128
// rows with one A plane, where 4 tiles of 128 rows would not leave room for the W prefetch in
// the 256 registers of two waves per SIMD); narrow N uses 1 and splits K until the grid covers
// the chip once (measured on 64 x 4096 x 4096 with
// the weights out of cache, reduction included: 29.6 us at one workgroup per CU, 33.0 us at
// two, 41.2 us at four).
struct SkPlan {
  bool use = false;
  int ntw = 4, ksplit = 1, kper = 0;
};

// Waves per workgroup: 128-row A chunks as hi and lo planes (double-buffered) leave LDS room
// for the epilogue staging of 4 waves only; one plane leaves room for all 8.
constexpr int sk_waves(int M, bool a_lo) { return M > 64 && a_lo ? 4 : SK_NW; }

SkPlan skinny_plan(int M, int N, int K, bool a_lo, bool w_lo, int cus) {
  SkPlan p;
  if (M > 128 || w_lo || K % SK_STEP != 0 || N % 4 != 0) return p;
  p.use = true;
  const int nw = sk_waves(M, a_lo);
  const int want = cus;
  const int wide = M > 64 && !a_lo ? 2 : 4;
  int tiles = (N + nw * 16 * wide - 1) / (nw * 16 * wide);
  p.ntw = wide;
  if (tiles < want) {
    p.ntw = 1;
    tiles = (N + nw * 16 - 1) / (nw * 16);
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
  constexpr int NW = sk_waves(16 * MT, ALO);
  using S = SkCfg<MT, NTW, NW, ALO>;
  // the residual is added by the reduction when K is split
  auto kern = (g.R && p.ksplit == 1 && !PK) ? skinny_kernel<MT, NTW, NW, ALO, PK, !PK>
                                            : skinny_kernel<MT, NTW, NW, ALO, PK, false>;
  const int nitems = ((g.N + S::BN - 1) / S::BN) * p.ksplit;
  // one workgroup per CU walks several items when there are more items than CUs
  const int grid = p.ksplit == 1 && nitems > device_cus() ? device_cus() : nitems;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(S::NT), 0, s, g, p.kper, nitems);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.ksplit == 1) return e;
  const size_t total = (size_t)g.M * g.N;
  const bool vec = g.N % 4 == 0 && (!g.C || g.ldc % 4 == 0) && (!g.R || g.ldr % 4 == 0) &&
                   (!(g.C_hi || g.C_h16) || g.ldch % 4 == 0);
  size_t blocks = ((vec ? total / 4 : total) + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (vec) hipLaunchKernelGGL(skinny_reduce4, dim3((unsigned)blocks), dim3(256), 0, s, g, p.ksplit);
  else hipLaunchKernelGGL(skinny_reduce, dim3((unsigned)blocks), dim3(256), 0, s, g, p.ksplit);
  return hipGetLastError();
}

template <int MT, bool ALO>
hipError_t launch_skinny_m(const GemmArgs& g, const SkPlan& p, hipStream_t s) {
  if constexpr (MT == 8 && !ALO) {
    if (p.ntw == 2) return g.w_packed ? launch_skinny_t<MT, 2, ALO, true>(g, p, s) : launch_skinny_t<MT, 2, ALO, false>(g, p, s);
  }
  if (g.w_packed) return p.ntw == 4 ? launch_skinny_t<MT, 4, ALO, true>(g, p, s) : launch_skinny_t<MT, 1, ALO, true>(g, p, s);
  return p.ntw == 4 ? launch_skinny_t<MT, 4, ALO, false>(g, p, s) : launch_skinny_t<MT, 1, ALO, false>(g, p, s);
}

template <bool ALO>
hipError_t launch_skinny_a(const GemmArgs& g, const SkPlan& p, hipStream_t s) {
  if (g.M <= 16) return launch_skinny_m<1, ALO>(g, p, s);
  if (g.M <= 32) return launch_skinny_m<2, ALO>(g, p, s);
  if (g.M <= 64) return launch_skinny_m<4, ALO>(g, p, s);
  return launch_skinny_m<8, ALO>(g, p, s);
}

// ------------------------------------------------------------- pipelined dense path
//
// Many rows (M >= 128): 128 x 128 output tiles, 4 waves of 64 x 64 (v_mfma_f32_32x32x16_bf16).
// A and W k-tiles (KT = 64 or 32 wide) go straight from global memory into LDS
// (global_load_lds_dwordx4), ST stages deep, so ST-1 tiles are in flight while one is
// multiplied; every LDS stage is its own object so that the compiler's wait for outstanding
// LDS DMA names only the stage being read.  Rows past M or N re-read the last valid row (their
// results are never stored); K must be a multiple of KT.  With KT = 32 a workgroup needs at
// most 72 KB of LDS, so two share a CU and each covers the other's waits for memory.

template <int TM, int TN, bool ALO, int ST, int KT>
struct DmaCfg {
  static constexpr int NT = 256;
  static constexpr int BM = 2 * TM * 32, BN = 2 * TN * 32;
  static constexpr int CPRT = KT / 8;                               // 16-byte units per tile row
  static constexpr int SA = BM * KT, SW = BN * KT;                  // elements per plane per stage
  static constexpr int STAGE = SA * (ALO ? 2 : 1) + SW;
  static constexpr int A_I = BM * CPRT / NT, W_I = BN * CPRT / NT; // DMA instructions per wave
  static constexpr int NI = A_I * (ALO ? 2 : 1) + W_I;
  static constexpr int VM = (ST - 2) * NI;
  static_assert(KT == 64 || KT == 32, "k-tile");
  static_assert(BM * CPRT % NT == 0 && BN * CPRT % NT == 0 && VM < 64 && ST >= 2 && ST <= 4, "dma gemm shape");
};

// LDS unit (16 bytes) of logical chunk `chunk` of tile row `row` in a KT-wide tile.  Rows of
// 128 bytes (KT = 64) XOR the chunk with (row / 2) mod 8, rows of 64 bytes (KT = 32) with
// (row / 4) mod 4: either way the 16 rows read by each 16-lane group of a fragment load fall
// on 16 distinct 16-byte bank groups.
template <int KT>
__device__ __forceinline__ int swz_key_t(int row) {
  if constexpr (KT == 64) return (row >> 1) & 7;
  else return (row >> 2) & 3;
}
template <int KT>
__device__ __forceinline__ int swz_t(int row, int chunk) {
  return row * (KT / 8) + (chunk ^ swz_key_t<KT>(row));
}

__device__ __forceinline__ void dma16(const bf16* src, bf16* lds) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
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

template <int TM, int TN, bool ALO, int ST, int KT>
__global__ void __launch_bounds__(256) gemm_dma_kernel(GemmArgs g) {
  using C = DmaCfg<TM, TN, ALO, ST, KT>;
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

  const int rows_a = min(C::BM, g.M - m0);
  const bf16* A0 = g.A_hi + (size_t)m0 * g.lda;
  const bf16* Al0 = (ALO ? g.A_lo : g.A_hi) + (size_t)m0 * g.lda;
  // W row segment of this tile (tiles never straddle a segment boundary)
  const bf16* wbase = g.W_hi;
  int wseg0 = 0, wseg1 = g.N;
  if (g.W2) {
    if (n0 >= g.N1 + g.N2) { wbase = g.W3; wseg0 = g.N1 + g.N2; }
    else if (n0 >= g.N1) { wbase = g.W2; wseg0 = g.N1; wseg1 = g.N1 + g.N2; }
    else wseg1 = g.N1;
  }
  const int rows_w = min(C::BN, wseg1 - n0);

  // unit u (16 bytes) of a stage plane: row u / CPRT, stored chunk u % CPRT = logical chunk ^
  // swz_key_t(row).  Source offsets of k-tile 0 per lane; k-tile t adds t * (a_step, w_step).
  size_t a_off[C::A_I], w_off[C::W_I];
#pragma unroll
  for (int i = 0; i < C::A_I; ++i) {
    const int u = (i * 4 + wave) * 64 + lane, row = u / C::CPRT;
    const int k = 8 * ((u % C::CPRT) ^ swz_key_t<KT>(row));
    a_off[i] = (size_t)min(row, rows_a - 1) * g.lda + k;
  }
#pragma unroll
  for (int i = 0; i < C::W_I; ++i) {
    const int u = (i * 4 + wave) * 64 + lane, row = u / C::CPRT;
    const int k = 8 * ((u % C::CPRT) ^ swz_key_t<KT>(row));
    const int n = n0 + min(row, rows_w - 1);
    w_off[i] = (size_t)(n - wseg0) * g.ldw + k;
  }
  const size_t w_step = (size_t)KT;
  auto issue = [&](int t, bf16* L, bf16* LW) {
    const size_t ka = (size_t)t * KT, kw = (size_t)t * w_step;
#pragma unroll
    for (int i = 0; i < C::A_I; ++i) {
      const int u0 = (i * 4 + wave) * 64;
      dma16(A0 + a_off[i] + ka, L + u0 * 8);
      if constexpr (ALO) dma16(Al0 + a_off[i] + ka, L + C::SA + u0 * 8);
    }
#pragma unroll
    for (int i = 0; i < C::W_I; ++i) dma16(wbase + w_off[i] + kw, LW + (i * 4 + wave) * 64 * 8);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  // Fragments of k-step ks + 1 are read while the MFMAs of k-step ks run.
  auto compute = [&](const bf16* L, const bf16* LW) {
    const bf16* sA = L;
    const bf16* sAl = L + C::SA;
    const bf16* sW = LW;
    bf16x8 fa[2][TM], fal[2][ALO ? TM : 1], fw[2][TN];
    auto frags = [&](int ks, int buf) {
      const int ch = 2 * ks + (lane >> 5);
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const int r = (wm * TM + a) * 32 + (lane & 31);
        fa[buf][a] = *reinterpret_cast<const bf16x8*>(sA + 8 * swz_t<KT>(r, ch));
        if constexpr (ALO) fal[buf][a] = *reinterpret_cast<const bf16x8*>(sAl + 8 * swz_t<KT>(r, ch));
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int r = (wn * TN + b) * 32 + (lane & 31);
        fw[buf][b] = *reinterpret_cast<const bf16x8*>(sW + 8 * swz_t<KT>(r, ch));
      }
    };
    frags(0, 0);
#pragma unroll
    for (int ks = 0; ks < KT / 16; ++ks) {
      if (ks + 1 < KT / 16) frags(ks + 1, (ks + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);   // the next k-step's LDS reads go out before these MFMAs
      const int cb = ks & 1;
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          acc[a][b] = mma32(fa[cb][a], fw[cb][b], acc[a][b]);
          if constexpr (ALO) acc[a][b] = mma32(fal[cb][a], fw[cb][b], acc[a][b]);
        }
    }
  };

  const int nk = (g.K + KT - 1) / KT;
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

template <int TM, int TN, bool ALO, int ST, int KT>
hipError_t launch_dma(const GemmArgs& g, hipStream_t s) {
  using C = DmaCfg<TM, TN, ALO, ST, KT>;
  const int tiles = ((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  hipLaunchKernelGGL((gemm_dma_kernel<TM, TN, ALO, ST, KT>), dim3(tiles), dim3(C::NT), 0, s, g);
  return hipGetLastError();
}

#ifndef HSPEC_DMA_KT
#define HSPEC_DMA_KT 32
#endif
// The dense products of the step (M = B k rows): 128 x 128 tiles, KT-wide k-tiles.
hipError_t launch_dense(const GemmArgs& g, hipStream_t s) {
  if constexpr (HSPEC_DMA_KT == 32)
    return g.A_lo ? launch_dma<2, 2, true, 3, 32>(g, s) : launch_dma<2, 2, false, 4, 32>(g, s);
  else
    return g.A_lo ? launch_dma<2, 2, true, 3, 64>(g, s) : launch_dma<2, 2, false, 4, 64>(g, s);
}

// ---------------------------------------------------------------------------------------
// Large products (M >= 256, the block positions of many requests).  Eight waves in a 2 x 4
// grid; a wave owns TM x TN blocks of 32 x 32 (v_mfma_f32_32x32x16_bf16) and reads 0.75 KB of
// LDS fragments per MFMA: 128 x 64 per wave (256 x 256 tiles) for a bf16 A, 64 x 64 per wave
// with the A lo plane (128 x 256 tiles, two products per block).  With 64 x 64 per wave and one
// plane the fragment reads alone would need the CU's whole LDS bandwidth at the MFMA rate.
// 32-wide k-tiles come into LDS by DMA, 4 stages deep.  The fragment reads run one k-step
// ahead across k-tiles: a tile's second k-step is read while its first is multiplied, and the
// next tile's first k-step while its second is, so the matrix unit has work queued across
// every wait for LDS or for the next tile.  With few tiles (tiles mod CUs small) the last tiles are split over K: unit
// u < full is whole tile u, the others are (tile, k-part) pairs whose fp32 partials a fix-up
// kernel sums in k-part order, so the result does not depend on scheduling.
#ifndef HSPEC_BIG_ST
#define HSPEC_BIG_ST 4
#endif
#ifndef HSPEC_BIG_MIN_M
#define HSPEC_BIG_MIN_M 256   // rows from which products take the large tiles
#endif
constexpr int GB_KT = 32, GB_NT = 512, GB_ST = HSPEC_BIG_ST;

// TMV: 32-row MFMA tiles per wave (block tiles of 64 TMV rows); hi/lo A takes 2 to fit registers.
template <bool ALO, int TMV = (ALO ? 2 : 4)>
struct BigCfg {
  static constexpr int TM = TMV, TN = 2;
  static constexpr int BM = 2 * TM * 32, BN = 4 * TN * 32;
  static constexpr int CPRT = GB_KT / 8;                           // 16-byte units per tile row
  static constexpr int SA = BM * GB_KT, SW = BN * GB_KT;           // elements per plane per stage
  static constexpr int A_I = BM * CPRT / GB_NT, W_I = BN * CPRT / GB_NT;   // DMA per wave
  static constexpr int NI = A_I * (ALO ? 2 : 1) + W_I;
  static_assert(BM * CPRT % GB_NT == 0 && BN * CPRT % GB_NT == 0 && (GB_ST - 3) * NI < 64 && GB_ST >= 3 &&
                GB_ST <= 5, "big gemm shape");
};

// Work division of a large product (host-computed, passed to the kernels).
struct BigPlan {
  int bm = 0, bn = 0;       // tile shape
  int mt = 0, nt = 0;       // tile grid
  int full = 0;             // units [0, full): whole tiles (virtual ids)
  int splits = 1, kper = 0; // remaining tiles: `splits` k-parts of kper k-tiles
  int units = 0;
};

template <bool ALO, int TMV>
__global__ void __launch_bounds__(GB_NT) gemm_big_kernel(GemmArgs g, BigPlan p) {
  using C = BigCfg<ALO, TMV>;
  constexpr int TM = C::TM, TN = C::TN, BM = C::BM, BN = C::BN;
  constexpr int PA = C::SA * (ALO ? 2 : 1);
  __shared__ __align__(16) bf16 A0s[PA], W0s[C::SW];
  __shared__ __align__(16) bf16 A1s[PA], W1s[C::SW];
  __shared__ __align__(16) bf16 A2s[PA], W2s[C::SW];
  __shared__ __align__(16) bf16 A3s[GB_ST > 3 ? PA : 8], W3s[GB_ST > 3 ? C::SW : 8];
  __shared__ __align__(16) bf16 A4s[GB_ST > 4 ? PA : 8], W4s[GB_ST > 4 ? C::SW : 8];
  auto sa_of = [&](auto I) -> bf16* {
    if constexpr (decltype(I)::value == 0) return A0s;
    else if constexpr (decltype(I)::value == 1) return A1s;
    else if constexpr (decltype(I)::value == 2) return A2s;
    else if constexpr (decltype(I)::value == 3) return A3s;
    else return A4s;
  };
  auto sw_of = [&](auto I) -> bf16* {
    if constexpr (decltype(I)::value == 0) return W0s;
    else if constexpr (decltype(I)::value == 1) return W1s;
    else if constexpr (decltype(I)::value == 2) return W2s;
    else if constexpr (decltype(I)::value == 3) return W3s;
    else return W4s;
  };

  // unit -> (tile, k-tile range)
  const int nk_all = g.K / GB_KT;
  int v, kb, ke;
  const int u = blockIdx.x;
  if (u < p.full) {
    int mt_, nt_;
    tile_of(u, p.full, p.mt, mt_, nt_);
    v = nt_ * p.mt + mt_;
    kb = 0;
    ke = nk_all;
  } else {
    const int r = u - p.full;
    v = p.full + r / p.splits;
    kb = (r % p.splits) * p.kper;
    ke = min(nk_all, kb + p.kper);
  }
  const int mt = v % p.mt, nt = v / p.mt;
  const int m0 = mt * BM, n0 = nt * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / 4, wn = wave % 4;

  const int rows_a = min(BM, g.M - m0);
  const bf16* A0 = g.A_hi + (size_t)m0 * g.lda;
  const bf16* Al0 = (ALO ? g.A_lo : g.A_hi) + (size_t)m0 * g.lda;
  const bf16* wbase = g.W_hi;   // W row segment of this tile (tiles never straddle one)
  int wseg0 = 0, wseg1 = g.N;
  if (g.W2) {
    if (n0 >= g.N1 + g.N2) { wbase = g.W3; wseg0 = g.N1 + g.N2; }
    else if (n0 >= g.N1) { wbase = g.W2; wseg0 = g.N1; wseg1 = g.N1 + g.N2; }
    else wseg1 = g.N1;
  }
  const int rows_w = min(BN, wseg1 - n0);

  // unit q (16 bytes) of a stage plane: row q / 4, stored chunk q % 4 = logical chunk ^ key(row).
  // Element offsets (32-bit: host-checked) from the tile's first row, at k-tile kb.
  const bf16* Ab = A0 + (size_t)kb * GB_KT;
  const bf16* Alb = Al0 + (size_t)kb * GB_KT;
  const bf16* Wb = wbase + (size_t)(n0 - wseg0) * g.ldw + (size_t)kb * GB_KT;
  int a_off[C::A_I], w_off[C::W_I];
#pragma unroll
  for (int i = 0; i < C::A_I; ++i) {
    const int q = (i * 8 + wave) * 64 + lane, row = q / C::CPRT;
    a_off[i] = min(row, rows_a - 1) * g.lda + 8 * ((q % C::CPRT) ^ swz_key_t<GB_KT>(row));
  }
#pragma unroll
  for (int i = 0; i < C::W_I; ++i) {
    const int q = (i * 8 + wave) * 64 + lane, row = q / C::CPRT;
    w_off[i] = min(row, rows_w - 1) * g.ldw + 8 * ((q % C::CPRT) ^ swz_key_t<GB_KT>(row));
  }
  auto issue = [&](int t, bf16* L, bf16* LW) {
    const int k = t * GB_KT;
#pragma unroll
    for (int i = 0; i < C::A_I; ++i) {
      const int q0 = (i * 8 + wave) * 64;
      dma16(Ab + (a_off[i] + k), L + q0 * 8);
      if constexpr (ALO) dma16(Alb + (a_off[i] + k), L + C::SA + q0 * 8);
    }
#pragma unroll
    for (int i = 0; i < C::W_I; ++i) dma16(Wb + (w_off[i] + k), LW + (i * 8 + wave) * 64 * 8);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  // fragment buffers: F0 holds k-step 0 of a tile, F1 k-step 1
  bf16x8 fa0[TM], fl0[ALO ? TM : 1], fw0[TN], fa1[TM], fl1[ALO ? TM : 1], fw1[TN];
  auto frags = [&](const bf16* L, const bf16* LW, int ks, bf16x8 (&fa)[TM], bf16x8 (&fl)[ALO ? TM : 1],
                   bf16x8 (&fw)[TN]) {
    const int ch = 2 * ks + (lane >> 5);
#pragma unroll
    for (int a = 0; a < TM; ++a) {
      const int r = (wm * TM + a) * 32 + (lane & 31);
      fa[a] = *reinterpret_cast<const bf16x8*>(L + 8 * swz_t<GB_KT>(r, ch));
      if constexpr (ALO) fl[a] = *reinterpret_cast<const bf16x8*>(L + C::SA + 8 * swz_t<GB_KT>(r, ch));
    }
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int r = (wn * TN + b) * 32 + (lane & 31);
      fw[b] = *reinterpret_cast<const bf16x8*>(LW + 8 * swz_t<GB_KT>(r, ch));
    }
  };
  auto mma = [&](const bf16x8 (&fa)[TM], const bf16x8 (&fl)[ALO ? TM : 1], const bf16x8 (&fw)[TN]) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        acc[a][b] = mma32(fa[a], fw[b], acc[a][b]);
        if constexpr (ALO) acc[a][b] = mma32(fl[a], fw[b], acc[a][b]);
      }
  };

  const int nk = ke - kb;
  // prologue without branches (tiles past the end re-read the last one into unused stages)
  [&]<int... I>(std::integer_sequence<int, I...>) {
    (issue(min(I, nk - 1), sa_of(Int<I>{}), sw_of(Int<I>{})), ...);
  }(std::make_integer_sequence<int, GB_ST - 1>{});
  wait_vmcnt<(GB_ST - 2) * C::NI>();   // tile 0 landed for this wave
  wg_barrier();
  frags(A0s, W0s, 0, fa0, fl0, fw0);

  // Step t (stage S = t mod ST): the MFMAs of k-step 0 of tile t are issued with the reads of
  // its k-step 1; tile t+1 is waited for (its DMA was issued ST-2 steps ago) and the stage of
  // tile t-1 (whose last reads every wave completed before this step's first MFMAs) refilled
  // with tile t+ST-1; then the MFMAs of k-step 1 with the reads of k-step 0 of tile t+1.
  // Scheduling groups place each fragment read right behind one MFMA (measured: the 1024 x
  // 16768 x 4096 product 187 -> 174 us, the 32000-row LM head 290 -> 267 us, other shapes
  // within 2 %), so the reads' latency runs under the batch instead of after it.
  auto interleave = [&]() {
    constexpr int nm = TM * TN * (ALO ? 2 : 1), nr = TM * (ALO ? 2 : 1) + TN;
    [&]<int... J>(std::integer_sequence<int, J...>) {
      (((void)J, __builtin_amdgcn_sched_group_barrier(0x008, 1, 0),   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0)), ...);      // one LDS read
    }(std::make_integer_sequence<int, (nr < nm ? nr : nm)>{});
    if constexpr (nm > nr) __builtin_amdgcn_sched_group_barrier(0x008, nm - nr, 0);
  };
  auto step = [&](int t, auto S, bool tail) {
    constexpr int s = decltype(S)::value, s1 = (s + 1) % GB_ST, sn = (s + GB_ST - 1) % GB_ST;
    mma(fa0, fl0, fw0);
    frags(sa_of(Int<s>{}), sw_of(Int<s>{}), 1, fa1, fl1, fw1);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    if (t + 1 < nk) {
      if (!tail) wait_vmcnt<(GB_ST - 3) * C::NI>();   // tiles t+2 .. t+ST-2 may stay in flight
      else wait_vmcnt<0>();
      wg_barrier();
      if (t + GB_ST - 1 < nk) issue(t + GB_ST - 1, sa_of(Int<sn>{}), sw_of(Int<sn>{}));
    }
    __builtin_amdgcn_sched_barrier(0);
    mma(fa1, fl1, fw1);
    // unconditional (a branch would split the scheduling region); after the last tile the
    // reads land in fragments nobody uses
    frags(sa_of(Int<s1>{}), sw_of(Int<s1>{}), 0, fa0, fl0, fw0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
  };
  int t0 = 0;
  // steady rounds: every DMA of the round's waits is issued (t + ST - 2 < nk for all its steps)
  for (; t0 + 2 * GB_ST - 2 < nk; t0 += GB_ST) {
    [&]<int... I>(std::integer_sequence<int, I...>) {
      (step(t0 + I, Int<I>{}, false), ...);
    }(std::make_integer_sequence<int, GB_ST>{});
  }
  for (; t0 < nk; t0 += GB_ST) {
    [&]<int... I>(std::integer_sequence<int, I...>) {
      ((t0 + I < nk ? step(t0 + I, Int<I>{}, true) : void()), ...);
    }(std::make_integer_sequence<int, GB_ST>{});
  }

  if (u < p.full) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
        store_block32(g, acc[a][b], m0 + (wm * TM + a) * 32, n0 + (wn * TN + b) * 32, lane);
  } else {
    // partial of k-part r % splits: [unit][BM][BN] fp32; lane holds rows 8(i/4)+4(l/32)+i%4
    float* part = g.part + (size_t)(u - p.full) * BM * BN;
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = (wm * TM + a) * 32 + 8 * (i / 4) + 4 * (lane >> 5) + (i % 4);
          part[r * BN + (wn * TN + b) * 32 + (lane & 31)] = acc[a][b][i];
        }
  }
}

// Sum of the k-parts of the split tiles in k-part order, then the usual epilogue.  One thread
// per 4 consecutive columns: 16-byte loads of the parts, 8 at a time, then of the residual;
// 16-byte stores.  VEC needs N, ldc, ldr and ldch % 4 == 0.
template <bool VEC>
__global__ void __launch_bounds__(256) gemm_big_fixup(GemmArgs g, BigPlan p) {
  constexpr int GROUP = 8;   // k-parts whose loads are issued together
  const int tiles = p.mt * p.nt - p.full;
  const size_t per = (size_t)p.bm * p.bn;
  const size_t quads = (size_t)tiles * per / 4;
  for (size_t q = (size_t)blockIdx.x * 256 + threadIdx.x; q < quads; q += (size_t)gridDim.x * 256) {
    const int tl = (int)(q / (per / 4));
    const int rc = (int)(q % (per / 4)) * 4;
    const int v = p.full + tl;
    const int m = (v % p.mt) * p.bm + rc / p.bn, n0 = (v / p.mt) * p.bn + rc % p.bn;
    if (m >= g.M || n0 >= g.N) continue;
    const float* src = g.part + (size_t)tl * p.splits * per + rc;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < p.splits; k0 += GROUP) {
      f32x4 part[GROUP];
#pragma unroll
      for (int k = 0; k < GROUP; ++k)
        part[k] = k0 + k < p.splits ? *reinterpret_cast<const f32x4*>(src + (size_t)(k0 + k) * per)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < GROUP; ++k) acc += part[k];   // absent parts add +0
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = n0 + e;
      if constexpr (!VEC) {
        if (n >= g.N) break;
        float s = acc[e];
        if (g.R) {
          s += g.r_bf16 ? bf2f(reinterpret_cast<const bf16*>(g.R)[(size_t)m * g.ldr + n])
                        : reinterpret_cast<const float*>(g.R)[(size_t)m * g.ldr + n];
        }
        if (g.C) g.C[(size_t)m * g.ldc + n] = s;
        if (g.C_hi) {
          const bf16 h = f2bf(s);
          g.C_hi[(size_t)m * g.ldch + n] = h;
          if (g.C_lo) g.C_lo[(size_t)m * g.ldch + n] = f2bf(s - bf2f(h));
        }
      }
    }
    if constexpr (VEC) {
      if (g.R) {
        if (g.r_bf16) {
          const bf16x4 r = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const bf16*>(g.R) + (size_t)m * g.ldr + n0);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += bf2f(r[e]);
        } else {
          acc += *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(g.R) + (size_t)m * g.ldr + n0);
        }
      }
      if (g.C) *reinterpret_cast<f32x4*>(g.C + (size_t)m * g.ldc + n0) = acc;
      if (g.C_hi) {
        bf16x4 h, l;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          h[e] = f2bf(acc[e]);
          l[e] = f2bf(acc[e] - bf2f(h[e]));
        }
        *reinterpret_cast<bf16x4*>(g.C_hi + (size_t)m * g.ldch + n0) = h;
        if (g.C_lo) *reinterpret_cast<bf16x4*>(g.C_lo + (size_t)m * g.ldch + n0) = l;
      }
    }
  }
}

// Whether the large-tile path serves a product, and its work division for `cus` CUs: whole
// tiles for every full round, the tiles of a short last round split over K so that the round
// fills the chip (at least 4 k-tiles per part).
bool big_ok(const GemmArgs& g) {
  if (g.M < HSPEC_BIG_MIN_M || g.W_lo || g.w_packed || g.K % GB_KT) return false;
  const int bm = g.A_lo ? BigCfg<true>::BM : BigCfg<false>::BM, bn = g.A_lo ? BigCfg<true>::BN : BigCfg<false>::BN;
  // 32-bit element offsets inside a tile's rows of A and W
  if ((long long)bm * g.lda >= (1ll << 31) || (long long)bn * g.ldw >= (1ll << 31)) return false;
  if (g.W2 && (g.N1 % bn || g.N2 % bn)) return false;
  return true;
}
// Row-tile height: 128 for hi/lo A; for one A plane 256, or 128 when 256-row tiles would not
// fill one round of CUs (then more whole tiles, fewer k-split ones).
int big_tm(int M, int N, bool a_lo, int cus) {
  if (a_lo) return 2;
  const int tiles256 = ((M + 255) / 256) * ((N + BigCfg<false>::BN - 1) / BigCfg<false>::BN);
  return tiles256 < cus ? 2 : 4;
}

BigPlan big_plan(int M, int N, int K, bool a_lo, int cus) {
  BigPlan p;
  p.bm = 64 * big_tm(M, N, a_lo, cus);
  p.bn = BigCfg<false>::BN;
  p.mt = (M + p.bm - 1) / p.bm;
  p.nt = (N + p.bn - 1) / p.bn;
  const int tiles = p.mt * p.nt, nk = K / GB_KT;
  const int rem = tiles % cus;
  int sp = rem ? cus / rem : 1;
  if (sp > nk / 4) sp = nk / 4;
  if (sp <= 1) {
    p.full = tiles;
    p.kper = nk;
  } else {
    p.full = tiles - rem;
    p.kper = (nk + sp - 1) / sp;
    p.splits = (nk + p.kper - 1) / p.kper;
  }
  p.units = p.full + (tiles - p.full) * p.splits;
  return p;
}
size_t big_scratch_elems(const BigPlan& p) {
  return (size_t)(p.mt * p.nt - p.full) * p.splits * p.bm * p.bn;
}

hipError_t launch_big(const GemmArgs& g, hipStream_t s) {
  BigPlan p = big_plan(g.M, g.N, g.K, g.A_lo != nullptr, device_cus());
  if (p.full < p.mt * p.nt && (!g.part || g.part_cap < big_scratch_elems(p))) {
    p.full = p.mt * p.nt;   // no room for partials: whole tiles only
    p.splits = 1;
    p.kper = g.K / GB_KT;
    p.units = p.full;
  }
  if (g.A_lo) hipLaunchKernelGGL((gemm_big_kernel<true, 2>), dim3(p.units), dim3(GB_NT), 0, s, g, p);
  else if (p.bm == 128) hipLaunchKernelGGL((gemm_big_kernel<false, 2>), dim3(p.units), dim3(GB_NT), 0, s, g, p);
  else hipLaunchKernelGGL((gemm_big_kernel<false, 4>), dim3(p.units), dim3(GB_NT), 0, s, g, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.full == p.mt * p.nt) return e;
  const size_t quads = big_scratch_elems(p) / p.splits / 4;
  size_t blocks = (quads + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  const bool vec = g.N % 4 == 0 && (!g.C || g.ldc % 4 == 0) && (!g.R || g.ldr % 4 == 0) && (!g.C_hi || g.ldch % 4 == 0);
  if (vec) hipLaunchKernelGGL(gemm_big_fixup<true>, dim3((unsigned)blocks), dim3(256), 0, s, g, p);
  else hipLaunchKernelGGL(gemm_big_fixup<false>, dim3((unsigned)blocks), dim3(256), 0, s, g, p);
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

__global__ void __launch_bounds__(256) pack_w_kernel(const bf16* __restrict__ W, int N, int K, _Float16* __restrict__ Wp) {
  // one 16-byte piece (row n, columns 8q..8q+7) per thread and iteration
  const int qr = K / 8, ntile = N / 16;
  const size_t total = (size_t)N * qr;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
    const int n = (int)(e / qr), q = (int)(e % qr);
    const int st = q / 4, c = q % 4, t = n / 16, i = n % 16;
    const int gr = t / 32, gs = min(32, ntile - 32 * gr);
    const size_t dst = ((size_t)gr * 32 * (K / 32) + (size_t)st * gs + (t - 32 * gr)) * 512 + (i + 16 * c) * 8;
    const u32x4 w = *reinterpret_cast<const u32x4*>(W + (size_t)n * K + 8 * q);
    f16x8 h;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // fp32 of the bf16 with its exponent raised by kPackScaleLog2 (bit arithmetic, so the scale
      // cannot be moved past the rounding to fp16).  Zeros and bf16 subnormals become +-0, inf
      // and NaN stay, and magnitudes of 2^16 and more (past fp16's range once scaled) become
      // +-inf without carrying into the sign bit.
      uint32_t b = ((w[e / 2] >> (16 * (e % 2))) & 0xffffu) << 16;
      const uint32_t ex = b & 0x7f800000u, sg = b & 0x80000000u;
      if (ex == 0) b = sg;
      else if (ex >= (uint32_t)(127 + 16) << 23 && ex != 0x7f800000u) b = sg | 0x7f800000u;
      else if (ex != 0x7f800000u) b += (uint32_t)kPackScaleLog2 << 23;
      h[e] = (_Float16)__uint_as_float(b);
    }
    *reinterpret_cast<f16x8*>(Wp + dst) = h;
  }
}

}  // namespace

hipError_t launch_pack_w(const bf16* W, int N, int K, _Float16* Wp, hipStream_t s) {
  if (N % 16 || K % SK_STEP || N <= 0 || K <= 0) return hipErrorInvalidValue;
  const size_t total = (size_t)N * (K / 8);
  size_t blocks = (total + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W, N, K, Wp);
  return hipGetLastError();
}

bool gemm_f16_out_ok(int M, int N, int K) {
  // the weight-streaming conditions (any CU count), in launches of at most 128 rows
  return M > 0 && skinny_plan(std::min(M, 128), N, K, false, false, 256).use && N % 4 == 0;
}

size_t gemm_scratch_elems(int M, int N, int K, bool a_lo, bool w_lo) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  // (past 128 rows the row-chunked weight-streaming launches run without a K split); the
  // plan for one A plane is covered too, since a caller sizing for hi/lo may pass one plane
  size_t n = 0;
  for (const bool lo : {a_lo, false}) {
    const SkPlan p = skinny_plan(M, N, K, lo, w_lo, device_cus());
    if (p.use && p.ksplit > 1) n = std::max(n, (size_t)p.ksplit * M * N);
  }
  if (M >= HSPEC_BIG_MIN_M && !w_lo && K % GB_KT == 0) {
    n = std::max(n, big_scratch_elems(big_plan(M, N, K, false, device_cus())));
    n = std::max(n, big_scratch_elems(big_plan(M, N, K, true, device_cus())));
  }
  return n;
}

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.f16 && !g.w_packed) return hipErrorInvalidValue;   // fp16 operands: the packed W only
  // products with the packed (fp16) W and fp16 outputs run on the weight-streaming path, in
  // launches of at most 128 rows
  if ((g.w_packed || g.C_h16) && g.M > 128 && !g.W2) {
    for (int m0 = 0; m0 < g.M; m0 += 128) {
      GemmArgs h = g;
      h.M = std::min(128, g.M - m0);
      h.A_hi += (size_t)m0 * g.lda;
      if (h.A_lo) h.A_lo += (size_t)m0 * g.lda;
      if (h.C) h.C += (size_t)m0 * g.ldc;
      if (h.C_hi) h.C_hi += (size_t)m0 * g.ldch;
      if (h.C_lo) h.C_lo += (size_t)m0 * g.ldch;
      if (h.C_h16) h.C_h16 += (size_t)m0 * g.ldch;
      if (h.C_l16) h.C_l16 += (size_t)m0 * g.ldch;
      if (h.R) h.R = h.r_bf16 ? (const void*)((const bf16*)h.R + (size_t)m0 * g.ldr)
                              : (const void*)((const float*)h.R + (size_t)m0 * g.ldr);
      if (hipError_t e = launch_gemm(h, s)) return e;
    }
    return hipSuccess;
  }
  if (g.W2) {
    if (big_ok(g)) return launch_big(g, s);
    const bool dma = g.M > 64 && !g.W_lo && !g.w_packed && g.K % BK == 0 && g.N1 % 128 == 0 && g.N2 % 128 == 0;
    if (dma) return launch_dense(g, s);
    // one launch per segment, each writing its own column range of C
    const bf16* ws[3] = {g.W_hi, g.W2, g.W3};
    const int n0s[3] = {0, g.N1, g.N1 + g.N2}, ns[3] = {g.N1, g.N2, g.N - g.N1 - g.N2};
    for (int i = 0; i < 3; ++i) {
      GemmArgs h = g;
      h.W2 = h.W3 = nullptr;
      h.W_hi = ws[i];
      h.N = ns[i];
      if (h.C) h.C += n0s[i];
      if (h.C_hi) h.C_hi += n0s[i];
      if (h.C_lo) h.C_lo += n0s[i];
      if (h.R) h.R = h.r_bf16 ? (const void*)((const bf16*)h.R + n0s[i]) : (const void*)((const float*)h.R + n0s[i]);
      if (hipError_t e = launch_gemm(h, s)) return e;
    }
    return hipSuccess;
  }
  SkPlan p = skinny_plan(g.M, g.N, g.K, g.A_lo != nullptr, g.W_lo != nullptr, device_cus());
  if ((g.C && g.ldc % 4) || ((g.C_hi || g.C_h16) && g.ldch % 4) || (g.R && g.ldr % 4)) p.use = false;   // 16-byte stores
  if (g.C_h16 && (!p.use || g.W2)) return hipErrorInvalidValue;   // only the weight-streaming path writes fp16
  if (g.C_l16 && !g.C_h16) return hipErrorInvalidValue;
  if (g.w_packed && (!p.use || g.N % 16 || g.K % BK || g.W_lo || g.R)) return hipErrorInvalidValue;   // packed W: no residual
  // packed W: one output, fp32 C or one fp16 plane (16-byte rows), not both, no bf16 planes
  if (g.w_packed && ((g.C != nullptr) == (g.C_h16 != nullptr) || g.C_hi || g.C_lo || g.C_l16 || (g.C_h16 && g.ldch % 8)))
    return hipErrorInvalidValue;
  if (p.use) {
    if (p.ksplit > 1 && (!g.part || g.part_cap < (size_t)p.ksplit * g.M * g.N)) {
      p.ksplit = 1;
      p.kper = ((g.K + SK_KC - 1) / SK_KC) * SK_KC;
    }
    return g.A_lo ? launch_skinny_a<true>(g, p, s) : launch_skinny_a<false>(g, p, s);
  }
  if (g.M <= 64 && !g.w_packed) return launch_cfg<1, 4, 2, 2>(g, s);      // 64 x 256: weight streaming
  if (big_ok(g)) return launch_big(g, s);
  if (!g.W_lo && g.K % BK == 0) return launch_dense(g, s);
  if (g.M <= 128) return launch_cfg<2, 2, 2, 4>(g, s);     // 128 x 256
  return launch_cfg<2, 2, 2, 2>(g, s);                     // 128 x 128: dense
}

}  // namespace hspec
