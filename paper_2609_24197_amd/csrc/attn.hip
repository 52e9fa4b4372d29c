// Block queries over one target layer's paged K/V cache, reused in place, plus the block's
// own K/V (H-Spec Sec. 3.3.2): the KV sweep over the cache, split along the context, and the
// reduction that combines the splits (and, in the precise mode, adds the block keys).
//
// Work unit = (request b, split s, KV head h).  Its query tile is the k*g rows of the block
// positions j and the g query heads of the group, stored as columns c = j*g + i; each wave
// owns 16 of those columns.  A persistent grid takes units from a device queue (the work list
// orders requests by decreasing split length).  Per unit, 32-key K/V
// tiles of the cache stream into LDS by direct DMA in a 3-stage pipeline:
//   * K tiles are read back as MFMA fragments, giving S^T = K Q^T with
//     v_mfma_f32_16x16x32_bf16, so each lane holds 4 keys of one column;
//   * the online softmax (base 2, lazily rescaled) reduces a column over its 4 lanes;
//   * the probabilities already sit in the B-fragment layout of O^T = V^T P^T, and V is read
//     transposed from LDS (ds_read_b64_tr_b16) as the A-fragment.
// The k block keys are taken one of two ways.  By default the last split of each request
// streams them after its cache keys, in bf16 like the cache, and a request with one split
// writes its output directly.  With block_in_sweep off (HSPEC_ATTN_PRECISE_IO) every split
// writes (unnormalised O, running max, running sum) and the reduction computes the block keys'
// softmax terms in fp32 from the hi/lo planes of q, k and v: few keys with large weights, where
// bf16 rounding does not average out over a stack of layers.  Either way the splits are combined in a fixed order, so results are bitwise
// reproducible and independent of where pages live in the pool.  Cache slots at or past ctx_len and pages the table does not
// reference are never read; page ids outside the pool raise a device status bit and read as
// zeros.
#include <climits>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "worklist.h"

#ifndef HSPEC_SWEEP_WPE
#define HSPEC_SWEEP_WPE 2   // waves per SIMD the sweep's register budget is sized for
#endif
#ifndef HSPEC_SWEEP_AUX
#define HSPEC_SWEEP_AUX 2   // cache-policy bits of the cache K/V loads (2: non-temporal)
#endif

namespace hspec {

namespace {

typedef unsigned short u16;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
#define LDS_AS __attribute__((address_space(3)))
#define GLB_AS __attribute__((address_space(1)))

constexpr int MIN_PAGE = 16;                    // smallest supported page size
constexpr int MAX_PIDS = MAX_SPLIT / MIN_PAGE + 1;

// Logical cache position i of a request lives in page page_table[b, i / ps], at offset i mod ps
// within it: the target's paged cache is read in place (Sec. 3.3.2, in-place KV reuse).  The
// sweep and the slot-map kernel both address the cache through these three functions, so the
// bit-exact slot-map test covers the sweep's own index path.  ps is a power of two, 2^lps.
__device__ __forceinline__ int page_of(int i, int lps) { return i >> lps; }
__device__ __forceinline__ int page_first_slot(int pid, int lps) { return pid << lps; }
__device__ __forceinline__ int slot_in_page(int first_slot, int i, int lps) { return first_slot + (i & ((1 << lps) - 1)); }

// Tile shape of the sweep.  QB: 16-column query blocks per wave; NW waves per workgroup;
// KT keys per tile; ST LDS stages (ST - 1 tiles in flight while one is multiplied).
template <int D, int QB, int NW, int KT, int ST, bool LO>
struct Sweep {
  static constexpr int NT = 64 * NW;
  static constexpr int COLS = 16 * QB;                 // query columns per wave
  static constexpr int CPR = D / 8;                    // 16-byte chunks per K/V row
  static constexpr int PLANES = LO ? 2 : 1;
  static constexpr int DMA = KT * CPR / NT;            // LDS-DMA instructions per wave per tensor-plane
  static constexpr int NDMA = 2 * PLANES * DMA;        // per wave per tile
  static constexpr int TILE = KT * D;                  // elements per tensor-plane
  static constexpr int STAGE = 2 * PLANES * TILE;      // K planes then V planes
  static constexpr int VM = (ST - 2) * NDMA;           // DMA instructions allowed in flight
  static_assert(KT % 32 == 0 && DMA >= 1 && KT * CPR % NT == 0, "tile shape");
  static_assert(ST >= 2 && ST <= 8 && VM < 64, "stages");
};

// Element offset of (row, column d) in a swizzled K/V tile.  16-byte chunk c of row r lives at
// chunk slot c ^ f(r).  For 256-byte rows f(r) = 2 (r mod 8) + (r / 8 mod 2): the 16 rows read
// by one 16-lane K fragment load land on 16 different slots, and the 8 rows x 32 bytes read by
// each half-wave of a transposing V load land on 8 different slot pairs, so neither access
// pattern has bank conflicts.  Shorter rows use c ^ (r mod CPR).
template <int CPR>
__device__ __forceinline__ int tile_off(int row, int d) {
  int f;
  if constexpr (CPR == 16) f = ((row & 7) << 1) | ((row >> 3) & 1);
  else f = row & (CPR - 1);
  return (row * CPR + ((d >> 3) ^ f)) * 8 + (d & 7);
}

// Running-max slack (log2 units): the softmax reference max is only raised, and O rescaled,
// when a tile's max exceeds it by more than this; probabilities then stay below 2^8.
constexpr float RESCALE_SLACK = 8.f;

template <int D, int QB, int NW, int KT, int ST, bool LO>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(HSPEC_SWEEP_WPE)))
attn_sweep(AttnArgs a) {
  using C = Sweep<D, QB, NW, KT, ST, LO>;
  constexpr int NS = D / 32;             // d-steps of the QK^T contraction
  constexpr int NDB = D / 16;            // 16-wide d blocks of the output
  constexpr int NKT = KT / 16;           // 16-key tiles per tile
  // One LDS object per stage, so the compiler can tell a stage being read from the stages
  // whose DMA is still in flight; the explicit waits below order them.
  __shared__ __align__(16) bf16 st0[C::STAGE];
  __shared__ __align__(16) bf16 st1[C::STAGE];
  __shared__ __align__(16) bf16 st2[ST > 2 ? C::STAGE : 8];
  __shared__ __align__(16) bf16 st3[ST > 3 ? C::STAGE : 8];
  __shared__ __align__(16) bf16 st4[ST > 4 ? C::STAGE : 8];
  __shared__ __align__(16) bf16 st5[ST > 5 ? C::STAGE : 8];
  __shared__ __align__(16) bf16 st6[ST > 6 ? C::STAGE : 8];
  __shared__ __align__(16) bf16 st7[ST > 7 ? C::STAGE : 8];
  __shared__ int pids[MAX_PIDS];
  auto stage = [&](auto S) -> bf16* {
    constexpr int s = decltype(S)::value;
    if constexpr (s == 0) return st0;
    else if constexpr (s == 1) return st1;
    else if constexpr (s == 2) return st2;
    else if constexpr (s == 3) return st3;
    else if constexpr (s == 4) return st4;
    else if constexpr (s == 5) return st5;
    else if constexpr (s == 6) return st6;
    else return st7;
  };

  __shared__ int s_item;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  const int lps = 31 - __builtin_clz(a.ps);
  const int g = a.Hq / a.Hkv, T = a.T, R = T * g;
  const int n_items = min(a.status[1], a.B * a.max_splits * a.Hkv);   // work-list length, capped at its array

  // The work list's entries (one per (request, split)) are copied to LDS when they fit, so
  // that an item's start waits on no memory round trip for its entry.  Otherwise thread 0
  // copies each claimed item's entry to s_units[0]; either way the entry is read from LDS.
  constexpr int UNITS_LDS = NW >= 4 ? 512 : 1;
  __shared__ int4 s_units[UNITS_LDS];
  const int n_units = (n_items + a.Hkv - 1) / a.Hkv;
  const bool units_lds = NW >= 4 && n_units <= UNITS_LDS;
  if (units_lds)
    for (int u = tid; u < n_units; u += C::NT) s_units[u] = reinterpret_cast<const int4*>(a.units)[u];

  // Persistent workgroups pull (request, split, KV head) items, longest splits first.  A
  // workgroup's first item is its own index; later ones come from the queue counter, offset by
  // the grid.  The next item is claimed while the last round of the current one is multiplied.
  // thread 0: queue ticket claimed ahead (item = grid + ticket), INT_MIN for none
  int next = (int)blockIdx.x - (int)gridDim.x;
  for (;;) {
  __syncthreads();                    // the previous item is finished by every wave
  if (tid == 0) {
    const int it = (int)gridDim.x + (next != INT_MIN ? next : atomicAdd(a.status + 2, 1));
    s_item = it;
    if (!units_lds && it < n_items) s_units[0] = reinterpret_cast<const int4*>(a.units)[it / a.Hkv];
  }
  next = INT_MIN;
  __syncthreads();
  const int item = s_item;
  if (item >= n_items) break;
  const int4 unit_e = s_units[units_lds ? item / a.Hkv : 0];
  const int b = unit_e.x >> 16, sp = unit_e.x & 0xffff, h = item % a.Hkv;
  const int hc = a.kv_remap ? (int)((a.kv_map >> (4 * h)) & 15) : h;   // the cache head this KV head reads
  const int L = unit_e.y;   // validated by the work-list kernel
  const int qlen = unit_e.z, nsplit = unit_e.w;
  const int k0 = swept_lo(a, L) + sp * qlen;
  const int k1 = min(L, k0 + qlen);
  const int kstart = k0;
  const int n_cache = kstart < k1 ? (k1 - kstart + KT - 1) / KT : 0;
  // the block keys follow the cache keys of a request's last split, unless the reduction takes them
  const int n_block = (a.block_in_sweep && sp == nsplit - 1) ? (T + KT - 1) / KT : 0;
  const int ntiles = n_cache + n_block;

  // query fragments: B operand of S^T = K Q^T (lane: column l16, dims 32 s + 8 g4 ..) and the
  // key window [lo, hi) of each column for cache keys and for block keys
  bf16x8 qf[QB][NS], qfl[QB][LO ? NS : 1];
  int c_lo[QB], c_hi[QB], b_hi[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int c = wave * C::COLS + qb * 16 + l16;
    const bool real = c < R;
    const int j = real ? c / g : 0;
    const int hq = h * g + (real ? c % g : 0);
    const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + 8 * g4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[qb][s] = real ? ld8(a.q_hi + off + 32 * s) : zero8();
      if constexpr (LO) qfl[qb][s] = real ? ld8(a.q_lo + off + 32 * s) : zero8();
    }
    c_lo[qb] = a.window > 0 ? L + j - a.window + 1 : INT_MIN;
    c_hi[qb] = real ? k1 : INT_MIN;
    b_hi[qb] = real ? (a.causal ? j + 1 : T) : INT_MIN;
  }
  // page ids of this split, validated once
  const int pg0 = page_of(k0, lps);
  if (n_cache > 0) {
    const int npg = page_of(k1 - 1, lps) - pg0 + 1;
    const int32_t* ptab = a.page_table + (size_t)b * a.max_pages + pg0;
    for (int e = tid; e < npg; e += C::NT) {
      int pid = ptab[e];
      if (pid < 0 || pid >= a.num_pages) {
        set_status(a.status, ST_BAD_PAGE);
        pid = 0;
      }
      pids[e] = page_first_slot(pid, lps);
    }
  }

  __syncthreads();   // page ids visible (LDS writes waited for, unlike the pipeline barrier)

  // LDS-DMA of tile ti into stage sb: wave w fills chunk slots [w*DMA*64, (w+1)*DMA*64) of
  // every tensor-plane; each lane picks the global chunk that belongs at its slot.  Keys past
  // the valid range load a valid row instead (finite values; masked out of the softmax).
  auto issue = [&](int ti, bf16* sb) {
    const bool cache = ti < n_cache;
    const int base = cache ? kstart + ti * KT : (ti - n_cache) * KT;
#pragma unroll
    for (int i = 0; i < C::DMA; ++i) {
      const int slot = (wave * C::DMA + i) * 64 + lane;
      const int row = slot / C::CPR;
      const int cl = (tile_off<C::CPR>(row, 8 * (slot % C::CPR)) / 8 - row * C::CPR);   // chunk stored here
      size_t off;
      int key = base + row;
      if (cache) {
        key = key < k1 ? key : k0;
        const int slot_id = slot_in_page(pids[page_of(key, lps) - pg0], key, lps);
        off = (size_t)slot_id * (a.Hkv_cache * D) + (hc * D + 8 * cl);
      } else {
        key = key < T ? key : 0;
        off = ((size_t)(b * T + key) * a.Hkv + h) * D + 8 * cl;
      }
      const bf16* Kp = cache ? a.kc_hi : a.kb_hi;
      const bf16* Vp = cache ? a.vc_hi : a.vb_hi;
      bf16* dst = sb + (wave * C::DMA + i) * 64 * 8;
      // the cache is read once per step: non-temporal loads (HSPEC_SWEEP_AUX cache-policy bits)
      __builtin_amdgcn_global_load_lds((const GLB_AS void*)(Kp + off), (LDS_AS void*)dst, 16, 0, HSPEC_SWEEP_AUX);
      __builtin_amdgcn_global_load_lds((const GLB_AS void*)(Vp + off), (LDS_AS void*)(dst + C::PLANES * C::TILE),
                                       16, 0, HSPEC_SWEEP_AUX);
      if constexpr (LO) {
        const bf16* Kl = cache ? a.kc_lo : a.kb_lo;
        const bf16* Vl = cache ? a.vc_lo : a.vb_lo;
        __builtin_amdgcn_global_load_lds((const GLB_AS void*)(Kl + off), (LDS_AS void*)(dst + C::TILE), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((const GLB_AS void*)(Vl + off),
                                         (LDS_AS void*)(dst + C::PLANES * C::TILE + C::TILE), 16, 0, 0);
      }
    }
  };

  f32x4 o[NDB][QB];
#pragma unroll
  for (int d = 0; d < NDB; ++d)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) o[d][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
  }
  const int lo_last = a.window > 0 ? L + (T - 1) - a.window + 1 : 0;

  auto compute = [&](int ti, const bf16* sb) {
    const bf16* sK = sb;
    const bf16* sV = sb + C::PLANES * C::TILE;
    const bool cache = ti < n_cache;
    const int base = cache ? kstart + ti * KT : (ti - n_cache) * KT;

    // all K fragments first, then the QK^T chains interleaved across key tiles
    bf16x8 kf[NKT][NS], kfl[NKT][LO ? NS : 1];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int off = tile_off<C::CPR>(kt * 16 + l16, 32 * s + 8 * g4);
        kf[kt][s] = *reinterpret_cast<const bf16x8*>(sK + off);
        if constexpr (LO) kfl[kt][s] = *reinterpret_cast<const bf16x8*>(sK + C::TILE + off);
      }
    f32x4 st[NKT][QB];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) st[kt][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          st[kt][qb] = mma16(kf[kt][s], qf[qb][s], st[kt][qb]);
          if constexpr (LO) {
            st[kt][qb] = mma16(kfl[kt][s], qf[qb][s], st[kt][qb]);
            st[kt][qb] = mma16(kf[kt][s], qfl[qb][s], st[kt][qb]);
          }
        }

    // V^T fragments (transposing LDS reads), issued before the softmax to hide their latency
    bf16x8 vf[KT / 32][NDB], vfl[KT / 32][LO ? NDB : 1];
    {
      const int vrow = 4 * g4 + (l16 >> 2);
#pragma unroll
      for (int kp = 0; kp < KT / 32; ++kp)
#pragma unroll
        for (int d = 0; d < NDB; ++d) {
          const int dc = d * 16 + 4 * (l16 & 3);
          const int o0 = tile_off<C::CPR>(kp * 32 + vrow, dc), o1 = tile_off<C::CPR>(kp * 32 + vrow + 16, dc);
          const s16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(sV + o0));
          const s16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(sV + o1));
          vf[kp][d] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
          if constexpr (LO) {
            const s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(sV + C::TILE + o0));
            const s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(sV + C::TILE + o1));
            vfl[kp][d] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7));
          }
        }
    }

    const bool full = cache && base + KT <= k1 && (a.window <= 0 || base >= lo_last);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
      if (full) {
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            st[kt][qb][i] *= a.scale_log2;
            mx = fmaxf(mx, st[kt][qb][i]);
          }
      } else {
        const int lo = cache ? c_lo[qb] : INT_MIN;
        const int hi = cache ? c_hi[qb] : b_hi[qb];
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = base + kt * 16 + 4 * g4 + i;
            const float v = ((key >= lo) & (key < hi)) ? st[kt][qb][i] * a.scale_log2 : -INFINITY;
            st[kt][qb][i] = v;
            mx = fmaxf(mx, v);
          }
      }
      mx = wave_max16x4(mx);
      if (__any(mx > m_run[qb] + RESCALE_SLACK)) {   // raise the reference max, rescale O and l
        const float m_new = fmaxf(m_run[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - (m_new == -INFINITY ? 0.f : m_new));
        l_run[qb] *= alpha;
#pragma unroll
        for (int d = 0; d < NDB; ++d) o[d][qb] *= alpha;
        m_run[qb] = m_new;
      }
      const float m_use = m_run[qb] == -INFINITY ? 0.f : m_run[qb];
      float sum = 0.f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = __builtin_amdgcn_exp2f(st[kt][qb][i] - m_use);
          st[kt][qb][i] = e;
          sum += e;
        }
      l_run[qb] += wave_sum16x4(sum);
    }

    // O^T += V^T P^T, 32 keys at a time (V^T fragments were read before the softmax)
#pragma unroll
    for (int kp = 0; kp < KT / 32; ++kp) {
      bf16x8 pf[QB], pfl[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const float v = st[2 * kp + (jj >> 2)][qb][jj & 3];
          const bf16 hv = f2bf(v);
          pf[qb][jj] = hv;
          if constexpr (LO) pfl[qb][jj] = f2bf(v - bf2f(hv));
        }
#pragma unroll
      for (int d = 0; d < NDB; ++d) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[d][qb] = mma16(vf[kp][d], pf[qb], o[d][qb]);
        if constexpr (LO) {
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            o[d][qb] = mma16(vfl[kp][d], pf[qb], o[d][qb]);
            o[d][qb] = mma16(vf[kp][d], pfl[qb], o[d][qb]);
          }
        }
      }
    }
  };

  // One pipeline step on stage S: wait for its tile, refill the stage freed last step, compute.
  auto step = [&](int ti, auto S) {
    constexpr int s = decltype(S)::value;
    if (ti >= ntiles) return;
    if (ti + ST - 2 < ntiles) wait_vmcnt<C::VM>();   // the next ST-2 tiles may stay in flight
    else wait_vmcnt<0>();
    wg_barrier();   // every wave's DMA for ti landed; every wave is done with the previous stage
    if (ti + ST - 1 < ntiles) issue(ti + ST - 1, stage(Int<(s + ST - 1) % ST>{}));
    compute(ti, stage(S));
  };
  auto round = [&]<int... I>(int t0, std::integer_sequence<int, I...>) { (step(t0 + I, Int<I>{}), ...); };

  [&]<int... I>(std::integer_sequence<int, I...>) {
    ((I < ntiles ? issue(I, stage(Int<I>{})) : void()), ...);
  }(std::make_integer_sequence<int, ST - 1>{});
  for (int t0 = 0; t0 < ntiles; t0 += ST) {
    if (tid == 0 && t0 + ST >= ntiles)
      next = (int)atomicInc(reinterpret_cast<unsigned*>(a.status + 2), 0xffffffffu);
    round(t0, std::make_integer_sequence<int, ST>{});
  }

  // write: lane holds O[column l16][d = 16 d + 4 g4 + i].  A request whose one split already
  // holds every key writes its output; otherwise the split's unnormalised (O, m, l).
  const size_t unit = ((size_t)b * a.Hkv + h) * a.max_splits + sp;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int c = wave * C::COLS + qb * 16 + l16;
    if (c >= R) continue;
    if (a.block_in_sweep && nsplit == 1) {
      const float inv = 1.f / l_run[qb];
      const int j = c / g, hq = h * g + c % g;
      const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + 4 * g4;
#pragma unroll
      for (int d = 0; d < NDB; ++d) {
        f32x4 v = o[d][qb] * inv;
        if (a.o_f32) *reinterpret_cast<f32x4*>(a.o_f32 + off + 16 * d) = v;
        if (a.o_bf16) {
          bf16x4 hv = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
          *reinterpret_cast<bf16x4*>(a.o_bf16 + off + 16 * d) = hv;
          if (a.o_bf16_lo) {
            bf16x4 lv;
#pragma unroll
            for (int e = 0; e < 4; ++e) lv[e] = f2bf(v[e] - bf2f(hv[e]));
            *reinterpret_cast<bf16x4*>(a.o_bf16_lo + off + 16 * d) = lv;
          }
        }
      }
    } else {
      float* po = a.part_o + (unit * R + c) * D + 4 * g4;
#pragma unroll
      for (int d = 0; d < NDB; ++d) *reinterpret_cast<f32x4*>(po + 16 * d) = o[d][qb];
      if (g4 == 0) {
        a.part_ml[(unit * R + c) * 2 + 0] = m_run[qb];
        a.part_ml[(unit * R + c) * 2 + 1] = l_run[qb];
      }
    }
  }
  }   // item loop
}

// Work list of the sweep (build_worklist) as a kernel of its own: the first kernel of an
// attention call that has no earlier kernel to carry it.
constexpr int PLAN_THREADS = 256;
constexpr int PLAN_RANK_MAX = 4096;

__global__ void __launch_bounds__(PLAN_THREADS) attn_plan(AttnArgs a, int clear_words) {
  __shared__ WorklistLds<PLAN_RANK_MAX> lds;
  build_worklist<PLAN_RANK_MAX>(a, clear_words, lds);
}

// Split reduction and block keys.  One workgroup per (request, KV head, 16 query columns);
// thread t serves column t / 16.  The block keys are taken in fp32 (q, k and v rebuilt from
// their hi/lo planes), 16 at a time, staged once per workgroup in LDS: lane t % 16 scores key
// t % 16 against its column, the column's 16 lanes keep an online softmax, then each lane
// accumulates D/16 dims of P V.  The same lanes then add sum_s O_s 2^(m_s - m*) and
// sum_s l_s 2^(m_s - m*) over the splits in split order; o = (O_blk + sum) / (l_blk + sum).
constexpr int RED_COLS = 16;
constexpr int RED_THREADS = 256;
constexpr int RED_NS = 4;   // splits whose loads are all issued together; more take further rounds

__device__ __forceinline__ f32x4 ld4_planes(const bf16* hi, const bf16* lo, size_t off) {
  const bf16x4 hv = *reinterpret_cast<const bf16x4*>(hi + off);
  f32x4 v = {bf2f(hv[0]), bf2f(hv[1]), bf2f(hv[2]), bf2f(hv[3])};
  if (lo) {
    const bf16x4 lv = *reinterpret_cast<const bf16x4*>(lo + off);
    v += f32x4{bf2f(lv[0]), bf2f(lv[1]), bf2f(lv[2]), bf2f(lv[3])};
  }
  return v;
}


// Split reduction when the sweep took the block keys: one thread per (column, 4 dims), PER of
// them per thread; o = sum_s O_s 2^(m_s - m*) / sum_s l_s 2^(m_s - m*) in split order.  Every
// load of a thread is issued before its first store (the stores could alias the partials as
// far as the compiler knows, so a loop over the PER outputs would serialise them).  Requests
// with one split were written by the sweep.
template <int D>
__global__ void __launch_bounds__(RED_THREADS) attn_merge(AttnArgs a) {
  constexpr int nq = D / 4, PER = RED_COLS * nq / RED_THREADS;
  static_assert(PER >= 1 && RED_COLS * nq % RED_THREADS == 0, "merge shape");
  const int g = a.Hq / a.Hkv, T = a.T, R = T * g;
  const int cblocks = (R + RED_COLS - 1) / RED_COLS;
  const int bh = blockIdx.x / cblocks, c0 = (blockIdx.x % cblocks) * RED_COLS;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const int nsplit = a.req[2 * b];   // splits of the request (the work-list kernel's choice)
  if (nsplit == 1) return;
  const size_t unit0 = ((size_t)b * a.Hkv + h) * a.max_splits;
  int cc[PER], d4[PER];
  bool ok[PER];
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    const int it = threadIdx.x + p * RED_THREADS;
    ok[p] = c0 + it / nq < R;
    cc[p] = ok[p] ? c0 + it / nq : c0;   // c0 < R: a valid column for the masked lanes
    d4[p] = (it % nq) * 4;
  }
  float m[PER][RED_NS], l[PER][RED_NS];
  f32x4 o[PER][RED_NS];
  auto fetch = [&](int s0) {
#pragma unroll
    for (int p = 0; p < PER; ++p)
#pragma unroll
      for (int i = 0; i < RED_NS; ++i) {
        // unconditional loads from a valid unit, dropped where unused: a branch around a load
        // would make the merged value wait before the next load goes out
        const bool in = ok[p] && s0 + i < nsplit;
        const size_t u = (unit0 + s0 + (s0 + i < nsplit ? i : 0)) * R + cc[p];
        const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + u * 2);
        const f32x4 ov = *reinterpret_cast<const f32x4*>(a.part_o + u * D + d4[p]);
        m[p][i] = in ? ml.x : -INFINITY;
        l[p][i] = in ? ml.y : 0.f;
        o[p][i] = in ? ov : f32x4{0.f, 0.f, 0.f, 0.f};
      }
  };
  float mstar[PER];
#pragma unroll
  for (int p = 0; p < PER; ++p) mstar[p] = -INFINITY;
  if (nsplit <= RED_NS) {
    fetch(0);
#pragma unroll
    for (int p = 0; p < PER; ++p)
#pragma unroll
      for (int i = 0; i < RED_NS; ++i) mstar[p] = fmaxf(mstar[p], m[p][i]);
  } else {
    for (int sp = 0; sp < nsplit; ++sp)
#pragma unroll
      for (int p = 0; p < PER; ++p) mstar[p] = fmaxf(mstar[p], a.part_ml[((unit0 + sp) * R + cc[p]) * 2]);
  }
  float lsum[PER];
  f32x4 acc[PER];
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    lsum[p] = 0.f;
    acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int s0 = 0; s0 < nsplit; s0 += RED_NS) {
    if (nsplit > RED_NS) fetch(s0);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const float m_use = mstar[p] == -INFINITY ? 0.f : mstar[p];
#pragma unroll
      for (int i = 0; i < RED_NS; ++i) {
        const float e = exp2f(m[p][i] - m_use);
        lsum[p] += l[p][i] * e;
        acc[p] += o[p][i] * e;
      }
    }
  }
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    if (!ok[p]) continue;
    const f32x4 v = acc[p] * (1.f / lsum[p]);
    const int j = cc[p] / g, hq = h * g + cc[p] % g;
    const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + d4[p];
    if (a.o_f32) *reinterpret_cast<f32x4*>(a.o_f32 + off) = v;
    if (a.o_bf16) {
      bf16x4 hv = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
      *reinterpret_cast<bf16x4*>(a.o_bf16 + off) = hv;
      if (a.o_bf16_lo) {
        bf16x4 lv;
#pragma unroll
        for (int e = 0; e < 4; ++e) lv[e] = f2bf(v[e] - bf2f(hv[e]));
        *reinterpret_cast<bf16x4*>(a.o_bf16_lo + off) = lv;
      }
    }
  }
}

template <int D>
__global__ void __launch_bounds__(RED_THREADS) attn_reduce(AttnArgs a) {
  constexpr int DP = D + 4;      // padded fp32 row: float4 reads of 16 different rows hit distinct banks
  constexpr int DPL = D / 16;    // dims per lane in P V and the merge
  constexpr int KC = 16;         // block keys per chunk
  constexpr int P4 = D / 4;      // float4 pieces per row
  static_assert(RED_COLS == 16 && RED_THREADS == 256, "16 columns x 16 lanes");
  __shared__ __align__(16) float sQ[RED_COLS * DP];
  __shared__ __align__(16) float sK[KC * DP];
  __shared__ __align__(16) float sV[KC * DP];
  __shared__ float sP[RED_COLS][KC + 1];
  const int g = a.Hq / a.Hkv, T = a.T, R = T * g;
  const int cblocks = (R + RED_COLS - 1) / RED_COLS;
  const int bh = blockIdx.x / cblocks, c0 = (blockIdx.x % cblocks) * RED_COLS;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const int nsplit = a.req[2 * b];   // splits of the request (the work-list kernel's choice)
  const size_t unit0 = ((size_t)b * a.Hkv + h) * a.max_splits;
  const int tid = threadIdx.x, ci = tid >> 4, ln = tid & 15;
  const bool live = c0 + ci < R;
  const int c = live ? c0 + ci : c0;
  const int j = c / g, hq = h * g + c % g;
  const int nb = a.causal ? j + 1 : T;   // block keys this column sees
  const int d0 = ln * DPL;

  // the splits' running maxima, sums and partial outputs for this lane's dims (all loads in
  // flight together when there are at most RED_NS splits), issued before the block keys
  float m[RED_NS], l[RED_NS];
  f32x4 o[RED_NS][DPL / 4];
  auto fetch = [&](int s0) {
#pragma unroll
    for (int i = 0; i < RED_NS; ++i) {
      const bool in = s0 + i < nsplit;
      const size_t u = (unit0 + s0 + (in ? i : 0)) * R + c;
      m[i] = in ? a.part_ml[u * 2] : -INFINITY;
      l[i] = in ? a.part_ml[u * 2 + 1] : 0.f;
#pragma unroll
      for (int e = 0; e < DPL / 4; ++e)
        o[i][e] = in ? *reinterpret_cast<const f32x4*>(a.part_o + u * D + d0 + 4 * e) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  if (nsplit <= RED_NS) fetch(0);

  // q of the workgroup's columns (the last column repeated past R)
  for (int p = tid; p < RED_COLS * P4; p += RED_THREADS) {
    const int r = p / P4, d4 = (p % P4) * 4;
    const int cr = min(c0 + r, R - 1);
    const size_t qoff = ((size_t)(b * T + cr / g) * a.Hq + h * g + cr % g) * D + d4;
    *reinterpret_cast<f32x4*>(sQ + r * DP + d4) = ld4_planes(a.q_hi, a.q_lo, qoff);
  }
  float mb = -INFINITY, lb = 0.f;
  f32x4 ob[DPL / 4];
#pragma unroll
  for (int e = 0; e < DPL / 4; ++e) ob[e] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < T; s0 += KC) {
    __syncthreads();   // q staged; the previous chunk's tiles are no longer read
    for (int p = tid; p < KC * P4; p += RED_THREADS) {
      const int r = p / P4, d4 = (p % P4) * 4;
      const size_t koff = ((size_t)(b * T + min(s0 + r, T - 1)) * a.Hkv + h) * D + d4;
      *reinterpret_cast<f32x4*>(sK + r * DP + d4) = ld4_planes(a.kb_hi, a.kb_lo, koff);
      *reinterpret_cast<f32x4*>(sV + r * DP + d4) = ld4_planes(a.vb_hi, a.vb_lo, koff);
    }
    __syncthreads();
    float sc = 0.f;
#pragma unroll 8
    for (int d = 0; d < D; d += 4) {
      const f32x4 qv = *reinterpret_cast<const f32x4*>(sQ + ci * DP + d);
      const f32x4 kv = *reinterpret_cast<const f32x4*>(sK + ln * DP + d);
      sc += qv[0] * kv[0] + qv[1] * kv[1] + qv[2] * kv[2] + qv[3] * kv[3];
    }
    sc = s0 + ln < nb ? sc * a.scale_log2 : -INFINITY;
    float cm = sc;
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) cm = fmaxf(cm, __shfl_xor(cm, msk));
    const float mn = fmaxf(mb, cm);   // finite: key 0 is seen by every column
    const float alpha = exp2f(mb - mn), pr = exp2f(sc - mn);
    float ps = pr;
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) ps += __shfl_xor(ps, msk);
    lb = lb * alpha + ps;
    mb = mn;
    sP[ci][ln] = pr;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < DPL / 4; ++e) ob[e] *= alpha;
#pragma unroll 4
    for (int s = 0; s < KC; ++s) {
      const float pv = sP[ci][s];
#pragma unroll
      for (int e = 0; e < DPL / 4; ++e) ob[e] += *reinterpret_cast<const f32x4*>(sV + s * DP + d0 + 4 * e) * pv;
    }
  }

  float mstar = mb;
  if (nsplit <= RED_NS) {
#pragma unroll
    for (int i = 0; i < RED_NS; ++i) mstar = fmaxf(mstar, m[i]);
  } else {
    for (int sp = 0; sp < nsplit; ++sp) mstar = fmaxf(mstar, a.part_ml[((unit0 + sp) * R + c) * 2]);
  }
  const float eb = exp2f(mb - mstar);
  float lsum = lb * eb;
  f32x4 acc[DPL / 4];
#pragma unroll
  for (int e = 0; e < DPL / 4; ++e) acc[e] = ob[e] * eb;
  for (int s0 = 0; s0 < nsplit; s0 += RED_NS) {
    if (nsplit > RED_NS) fetch(s0);
#pragma unroll
    for (int i = 0; i < RED_NS; ++i) {
      const float w = exp2f(m[i] - mstar);
      lsum += l[i] * w;
#pragma unroll
      for (int e = 0; e < DPL / 4; ++e) acc[e] += o[i][e] * w;
    }
  }
  if (!live) return;
  const float inv = 1.f / lsum;
  const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + d0;
#pragma unroll
  for (int e = 0; e < DPL / 4; ++e) {
    const f32x4 v = acc[e] * inv;
    if (a.o_f32) *reinterpret_cast<f32x4*>(a.o_f32 + off + 4 * e) = v;
    if (a.o_bf16) {
      bf16x4 hv = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
      *reinterpret_cast<bf16x4*>(a.o_bf16 + off + 4 * e) = hv;
      if (a.o_bf16_lo) {
        bf16x4 lv;
#pragma unroll
        for (int q = 0; q < 4; ++q) lv[q] = f2bf(v[q] - bf2f(hv[q]));
        *reinterpret_cast<bf16x4*>(a.o_bf16_lo + off + 4 * e) = lv;
      }
    }
  }
}

__global__ void gather_slots_kernel(int B, int max_pages, int ps, int num_pages, const int32_t* pt,
                                    const int32_t* lens, int max_ctx_len, int32_t* slots, int* status) {
  const int b = blockIdx.y;
  const int lps = 31 - __builtin_clz(ps);
  int L = lens[b];
  int cap = max_pages * ps < max_ctx_len ? max_pages * ps : max_ctx_len;
  if (L < 0 || L > cap) {
    if (threadIdx.x == 0 && blockIdx.x == 0) set_status(status, ST_BAD_CTX_LEN);
    L = L < 0 ? 0 : cap;
  }
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < max_ctx_len; i += gridDim.x * blockDim.x) {
    int v = -1;
    if (i < L) {
      int pid = pt[(size_t)b * max_pages + page_of(i, lps)];
      if (pid < 0 || pid >= num_pages) set_status(status, ST_BAD_PAGE);
      else v = slot_in_page(page_first_slot(pid, lps), i, lps);
    }
    slots[(size_t)b * max_ctx_len + i] = v;
  }
}

#ifndef HSPEC_SWEEP_QB
#define HSPEC_SWEEP_QB 1
#endif
#ifndef HSPEC_SWEEP_ST
#define HSPEC_SWEEP_ST 3
#endif
#ifndef HSPEC_SWEEP_KT
#define HSPEC_SWEEP_KT 32   // keys per tile (at least; a multiple of 32)
#endif

// One compiled variant of the sweep: tile keys, pipeline depth and the kernel, from the head
// dim, the waves per workgroup and the storage (LO: fp32 as hi/lo planes).
template <int D, int QB, int NW, bool LO>
struct SweepVariant {
  static constexpr int KT0 = 512 * NW / D > 32 ? 512 * NW / D : 32;  // every lane DMAs at least one chunk
  static constexpr int KT = KT0 > HSPEC_SWEEP_KT ? KT0 : HSPEC_SWEEP_KT;
  static constexpr int NDMA = 2 * (LO ? 2 : 1) * KT * (D / 8) / (64 * NW);
  static constexpr int ST_MAX = 2 + 63 / NDMA;                       // vmcnt holds at most 63
  static constexpr int ST = LO ? 2 : (HSPEC_SWEEP_ST < ST_MAX ? HSPEC_SWEEP_ST : ST_MAX);
  static constexpr int THREADS = 64 * NW;
  static constexpr auto kern = attn_sweep<D, QB, NW, KT, ST, LO>;

  // Resident workgroups on the current device (the persistent grid), cached per device.
  static hipError_t slots(int& out) {
    static int slots_of[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    int& sl = slots_of[dev & 63];
    if (sl == 0) {
      int cus = 0, per_cu = 0;
      e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
      if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, THREADS, 0);
      if (e != hipSuccess) return e;
      sl = cus * (per_cu > 0 ? per_cu : 1);
    }
    out = sl;
    return hipSuccess;
  }
};

// Calls f(SweepVariant<...>{}) for the variant the arguments select; hipErrorInvalidValue if none.
// D: head dim; R: query rows per KV head (k g); lo: fp32 storage (the cache as hi/lo planes).
template <class F>
hipError_t with_sweep_variant(int D, int R, bool lo, F f) {
  constexpr int QB = HSPEC_SWEEP_QB;
  const int nw = (R + 16 * QB - 1) / (16 * QB);
  auto by_nw = [&](auto d, auto l) -> hipError_t {
    constexpr int Dv = decltype(d)::value;
    constexpr bool Lv = decltype(l)::value;
    if (nw <= 1) return f(SweepVariant<Dv, QB, 1, Lv>{});
    if (nw <= 2) return f(SweepVariant<Dv, QB, 2, Lv>{});
    if (nw <= 4) return f(SweepVariant<Dv, QB, 4, Lv>{});
    if (nw <= 8) return f(SweepVariant<Dv, QB, 8, Lv>{});
    return hipErrorInvalidValue;
  };
  // 65..128 rows with one storage plane: two 16-column blocks per wave, so that four waves
  // cover the rows and two workgroups share a CU (one workgroup of eight waves stalls the
  // whole CU at each tile barrier)
  if (!lo && QB == 1 && R > 64 && R <= 128) {
    if (D == 128) return f(SweepVariant<128, 2, 4, false>{});
    if (D == 64) return f(SweepVariant<64, 2, 4, false>{});
    return hipErrorInvalidValue;
  }
  if (D == 128) return lo ? by_nw(Int<128>{}, std::true_type{}) : by_nw(Int<128>{}, std::false_type{});
  if (D == 64) return lo ? by_nw(Int<64>{}, std::true_type{}) : by_nw(Int<64>{}, std::false_type{});
  return hipErrorInvalidValue;
}

}  // namespace

size_t attention_partials_bytes(int B, int Hkv, int max_splits, int R, int D) {
  const size_t units = (size_t)B * Hkv * max_splits;
  return units * R * D * sizeof(float) + units * R * 2 * sizeof(float);
}

int attention_sweep_grid(int D, int R, bool lo) {
  int grid = 0;
  const hipError_t e = with_sweep_variant(D, R, lo, [&](auto v) { return decltype(v)::slots(grid); });
  return e == hipSuccess ? grid : 0;
}

hipError_t launch_attention_plan(const AttnArgs& a, int clear_words, hipStream_t s) {
  hipLaunchKernelGGL(attn_plan, dim3(1), dim3(PLAN_THREADS), 0, s, a, clear_words);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s, unsigned parts) {
  hipError_t e = hipSuccess;
  if (parts & ATTN_SWEEP) {
    if (!a.q_hi || !a.kc_hi || !a.vc_hi) return hipErrorInvalidValue;
    if (a.block_in_sweep ? (!a.kb_hi || !a.vb_hi) : (!a.part_o || !a.part_ml)) return hipErrorInvalidValue;
    e = with_sweep_variant(a.D, a.T * (a.Hq / a.Hkv), a.kc_lo != nullptr, [&](auto v) -> hipError_t {
      using V = decltype(v);
      int slots = 0;
      const hipError_t es = V::slots(slots);
      if (es != hipSuccess) return es;
      const long long items = (long long)a.B * a.max_splits * a.Hkv;
      const int grid = (int)(items < slots ? items : slots);
      hipLaunchKernelGGL(V::kern, dim3(grid), dim3(V::THREADS), 0, s, a);
      return hipGetLastError();
    });
    if (e != hipSuccess) return e;
  }
  if (parts & ATTN_REDUCE) {
    const int R = a.T * (a.Hq / a.Hkv);
    const int cblocks = (R + RED_COLS - 1) / RED_COLS;
    if (a.block_in_sweep) {
      if (a.max_splits > 1) {
        if (!a.part_o || !a.part_ml) return hipErrorInvalidValue;
        if (a.D == 128) hipLaunchKernelGGL(attn_merge<128>, dim3(a.B * a.Hkv * cblocks), dim3(RED_THREADS), 0, s, a);
        else hipLaunchKernelGGL(attn_merge<64>, dim3(a.B * a.Hkv * cblocks), dim3(RED_THREADS), 0, s, a);
      }
      return hipGetLastError();
    }
    if (!a.q_hi || !a.kb_hi || !a.vb_hi || !a.part_o || !a.part_ml) return hipErrorInvalidValue;   // block q/k/v, partials
    if (a.D == 128) hipLaunchKernelGGL(attn_reduce<128>, dim3(a.B * a.Hkv * cblocks), dim3(RED_THREADS), 0, s, a);
    else hipLaunchKernelGGL(attn_reduce<64>, dim3(a.B * a.Hkv * cblocks), dim3(RED_THREADS), 0, s, a);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_gather_slots(int B, int max_pages, int ps, int num_pages, const int32_t* page_table,
                               const int32_t* ctx_lens, int max_ctx_len, int32_t* slots, int* status,
                               hipStream_t s) {
  if (B <= 0 || max_ctx_len <= 0) return hipSuccess;
  int bx = (max_ctx_len + 255) / 256;
  if (bx > 1024) bx = 1024;
  hipLaunchKernelGGL(gather_slots_kernel, dim3(bx, B), dim3(256), 0, s, B, max_pages, ps, num_pages,
                     page_table, ctx_lens, max_ctx_len, slots, status);
  return hipGetLastError();
}

}  // namespace hspec
