// Block queries over one target layer's paged K/V cache, reused in place, plus the block's
// own K/V (H-Spec Sec. 3.3.2): the KV sweep, split along the context, and the cross-split
// softmax reduction.
//
// Work unit = (request b, KV head h, split s).  Its query tile is the k*g rows of the block
// positions j and the g query heads of the group, stored as columns c = j*g + i.  Each wave
// owns 32 of those columns; the waves of a workgroup share 64-key K/V tiles staged in LDS:
//   * K tiles are read back as MFMA A-fragments (16 keys x 32 dims, 16-byte reads), giving
//     S^T = K Q^T with v_mfma_f32_16x16x32_bf16, so each lane holds 4 keys of one column;
//   * the online softmax reduces a column over its 4 lanes with two cross-lane shuffles;
//   * the probabilities already sit in the B-fragment layout of O^T = V^T P^T, and V is read
//     transposed from LDS (one bf16 per read) as the A-fragment.
// Global loads of the next tile are issued before the current tile is multiplied.  A split
// that covers a whole request writes the normalised output directly; otherwise it writes
// (unnormalised O, running max, running sum) and the reduction kernel combines the splits
// in a fixed order, so results are bitwise reproducible and independent of where pages
// live in the pool.  Cache slots at or past ctx_len and pages the table does not reference
// are never read; page ids outside the pool raise a device status bit and read as zeros.
#include "common.h"
#include "kernels.h"

namespace hspec {

namespace {

constexpr int KT = 64;   // keys per tile
typedef unsigned short u16;
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

template <int D>
struct AttnCfg {
  static constexpr int CPR = D / 8;              // 16-byte chunks per K/V row
  static constexpr int TILE = KT * D;            // elements per tile per plane
};

__device__ __forceinline__ int clamp_len(const AttnArgs& a, int b) {
  int L = a.ctx_lens[b];
  int cap = a.max_pages * a.ps;
  if (cap > a.max_ctx_len) cap = a.max_ctx_len;
  if (L < 0 || L > cap) {
    set_status(a.status, ST_BAD_CTX_LEN);
    L = L < 0 ? 0 : cap;
  }
  return L;
}

template <int D>
__device__ __forceinline__ int lds_idx(int row, int chunk) {
  return (row * AttnCfg<D>::CPR + (chunk ^ (row & (AttnCfg<D>::CPR - 1)))) * 8;
}

template <int D, int NW, bool LO>
__global__ void __launch_bounds__(64 * NW)
attn_sweep(AttnArgs a) {
  using C = AttnCfg<D>;
  constexpr int NT = 64 * NW;
  constexpr int CH = KT * C::CPR / NT;            // chunks per thread per tensor per plane
  constexpr int NS = D / 32;                      // d-steps of the QK^T contraction
  constexpr int NDB = D / 16;                     // 16-wide d blocks of the output
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* sK = reinterpret_cast<bf16*>(smem);
  bf16* sV = sK + C::TILE * (LO ? 2 : 1);

  const int sp = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int L = clamp_len(a, b);
  const int nsplit = L > 0 ? (L + a.split - 1) / a.split : 1;
  if (sp >= nsplit) return;
  const int g = a.Hq / a.Hkv, T = a.T, R = T * g;
  const int k0 = sp * a.split;
  const int k1 = min(L, k0 + a.split);
  const bool last = sp == nsplit - 1;
  int kstart = k0;
  if (a.window > 0) {
    int lo0 = L - a.window + 1;
    if (lo0 > kstart) kstart = k0 + ((lo0 - k0) / KT) * KT;
  }
  const int n_cache = kstart < k1 ? (k1 - kstart + KT - 1) / KT : 0;
  const int n_block = last ? (T + KT - 1) / KT : 0;
  const int ntiles = n_cache + n_block;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;

  // ---- query fragments: B operand of S^T = K Q^T (lane: column l16, dims 32s + 8 g4 ..)
  bf16x8 qf[2][NS], qfl[2][LO ? NS : 1];
  int colj[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int c = wave * 32 + qb * 16 + l16;
    colj[qb] = c < R ? c / g : T;          // padding columns: never valid, never written
    const int hq = h * g + (c < R ? c % g : 0);
    const size_t off = ((size_t)(b * T + (c < R ? c / g : 0)) * a.Hq + hq) * D + 8 * g4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[qb][s] = c < R ? ld8(a.q_hi + off + 32 * s) : zero8();
      if constexpr (LO) qfl[qb][s] = c < R ? ld8(a.q_lo + off + 32 * s) : zero8();
    }
  }

  f32x4 o[NDB][2];
#pragma unroll
  for (int d = 0; d < NDB; ++d)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) o[d][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

  // ---- cooperative tile loads (registers, then LDS)
  bf16x8 rk[CH], rv[CH], rkl[LO ? CH : 1], rvl[LO ? CH : 1];
  const int32_t* ptab = a.page_table + (size_t)b * a.max_pages;
  auto load_tile = [&](int ti) {
    const bool cache = ti < n_cache;
    const int base = cache ? kstart + ti * KT : (ti - n_cache) * KT;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int q = i * NT + tid, r = q / C::CPR, c = q % C::CPR;
      const int key = base + r;
      bool ok;
      size_t off = 0;
      if (cache) {
        ok = key < k1;
        if (ok) {
          int pid = ptab[key / a.ps];
          if (pid < 0 || pid >= a.num_pages) {
            set_status(a.status, ST_BAD_PAGE);
            ok = false;
          } else {
            off = ((size_t)(pid * a.ps + key % a.ps) * a.Hkv + h) * D + 8 * c;
          }
        }
      } else {
        ok = key < T;
        off = ((size_t)(b * T + key) * a.Hkv + h) * D + 8 * c;
      }
      const bf16* K = cache ? a.kc_hi : a.kb_hi;
      const bf16* V = cache ? a.vc_hi : a.vb_hi;
      rk[i] = ok ? ld8(K + off) : zero8();
      rv[i] = ok ? ld8(V + off) : zero8();
      if constexpr (LO) {
        const bf16* Kl = cache ? a.kc_lo : a.kb_lo;
        const bf16* Vl = cache ? a.vc_lo : a.vb_lo;
        rkl[i] = ok ? ld8(Kl + off) : zero8();
        rvl[i] = ok ? ld8(Vl + off) : zero8();
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int q = i * NT + tid, r = q / C::CPR, c = q % C::CPR;
      const int idx = lds_idx<D>(r, c);
      *reinterpret_cast<bf16x8*>(sK + idx) = rk[i];
      *reinterpret_cast<bf16x8*>(sV + idx) = rv[i];
      if constexpr (LO) {
        *reinterpret_cast<bf16x8*>(sK + C::TILE + idx) = rkl[i];
        *reinterpret_cast<bf16x8*>(sV + C::TILE + idx) = rvl[i];
      }
    }
  };

  const int lo_last = a.window > 0 ? L + (T - 1) - a.window + 1 : 0;
  if (ntiles > 0) load_tile(0);
  for (int ti = 0; ti < ntiles; ++ti) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (ti + 1 < ntiles) load_tile(ti + 1);

    const bool cache = ti < n_cache;
    const int base = cache ? kstart + ti * KT : (ti - n_cache) * KT;

    // S^T tile: 4 key-tiles of 16 x 2 column blocks of 16
    f32x4 st[4][2];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) st[kt][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int idx = lds_idx<D>(kt * 16 + l16, 4 * s + g4);
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(sK + idx);
        bf16x8 kfl;
        if constexpr (LO) kfl = *reinterpret_cast<const bf16x8*>(sK + C::TILE + idx);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          st[kt][qb] = mma16(kf, qf[qb][s], st[kt][qb]);
          if constexpr (LO) {
            st[kt][qb] = mma16(kfl, qf[qb][s], st[kt][qb]);
            st[kt][qb] = mma16(kf, qfl[qb][s], st[kt][qb]);
          }
        }
      }
    }

    // scale into log2 units, mask, online softmax per column
    const bool full = cache && base + KT <= k1 && (a.window <= 0 || base >= lo_last);
    float p[4][2][4];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int j = colj[qb];
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = st[kt][qb][i] * a.scale_log2;
          if (!full) {
            const int key = base + kt * 16 + 4 * g4 + i;
            bool ok;
            if (cache) ok = key < k1 && (a.window <= 0 || key >= L + j - a.window + 1);
            else ok = key < T && (!a.causal || key <= j);
            if (j >= T) ok = false;
            v = ok ? v : -INFINITY;
          }
          p[kt][qb][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = wave_max16x4(mx);
      const float m_new = fmaxf(m_run[qb], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run[qb] - m_use);
      float sum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = exp2f(p[kt][qb][i] - m_use);
          p[kt][qb][i] = e;
          sum += e;
        }
      sum = wave_sum16x4(sum);
      l_run[qb] = l_run[qb] * alpha + sum;
      m_run[qb] = m_new;
#pragma unroll
      for (int d = 0; d < NDB; ++d) o[d][qb] *= alpha;
    }

    // O^T += V^T P^T over two 32-key halves
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
      bf16x8 pf[2], pfl[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const float v = p[2 * kp + (jj >> 2)][qb][jj & 3];
          const bf16 hv = f2bf(v);
          pf[qb][jj] = hv;
          if constexpr (LO) pfl[qb][jj] = f2bf(v - bf2f(hv));
        }
#pragma unroll
      for (int d = 0; d < NDB; ++d) {
        const int dd = d * 16 + l16;
        u16x8 vv, vvl;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int key = kp * 32 + (jj < 4 ? 4 * g4 + jj : 16 + 4 * g4 + (jj - 4));
          const int idx = lds_idx<D>(key, dd >> 3) + (dd & 7);
          vv[jj] = reinterpret_cast<const u16*>(sV)[idx];
          if constexpr (LO) vvl[jj] = reinterpret_cast<const u16*>(sV + C::TILE)[idx];
        }
        const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          o[d][qb] = mma16(vf, pf[qb], o[d][qb]);
          if constexpr (LO) {
            o[d][qb] = mma16(__builtin_bit_cast(bf16x8, vvl), pf[qb], o[d][qb]);
            o[d][qb] = mma16(vf, pfl[qb], o[d][qb]);
          }
        }
      }
    }
  }

  // ---- write: lane holds O[column l16][d = 16 d + 4 g4 + i]
  const size_t unit = ((size_t)b * a.Hkv + h) * a.max_splits + sp;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int c = wave * 32 + qb * 16 + l16;
    if (c >= R) continue;
    if (nsplit == 1) {
      const float inv = 1.f / l_run[qb];
      const int j = c / g, hq = h * g + c % g;
      const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + 4 * g4;
#pragma unroll
      for (int d = 0; d < NDB; ++d) {
        f32x4 v = o[d][qb] * inv;
        if (a.o_f32) *reinterpret_cast<f32x4*>(a.o_f32 + off + 16 * d) = v;
        if (a.o_bf16) {
#pragma unroll
          for (int i = 0; i < 4; ++i) a.o_bf16[off + 16 * d + i] = f2bf(v[i]);
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
}

// One workgroup per (request, KV head): o = sum_s O_s 2^(m_s - m*) / sum_s l_s 2^(m_s - m*).
__global__ void __launch_bounds__(256) attn_reduce(AttnArgs a) {
  const int b = blockIdx.x / a.Hkv, h = blockIdx.x % a.Hkv;
  const int L = clamp_len(a, b);
  const int nsplit = L > 0 ? (L + a.split - 1) / a.split : 1;
  if (nsplit == 1) return;
  const int g = a.Hq / a.Hkv, T = a.T, R = T * g, D = a.D;
  const size_t unit0 = ((size_t)b * a.Hkv + h) * a.max_splits;
  const int nq = D / 4;
  for (int it = threadIdx.x; it < R * nq; it += blockDim.x) {
    const int c = it / nq, d4 = (it % nq) * 4;
    float mstar = -INFINITY;
    for (int s = 0; s < nsplit; ++s) mstar = fmaxf(mstar, a.part_ml[((unit0 + s) * R + c) * 2]);
    const float m_use = mstar == -INFINITY ? 0.f : mstar;
    float lsum = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < nsplit; ++s) {
      const float* ml = a.part_ml + ((unit0 + s) * R + c) * 2;
      const float w = exp2f(ml[0] - m_use);
      lsum += ml[1] * w;
      acc += *reinterpret_cast<const f32x4*>(a.part_o + ((unit0 + s) * R + c) * D + d4) * w;
    }
    acc *= 1.f / lsum;
    const int j = c / g, hq = h * g + c % g;
    const size_t off = ((size_t)(b * T + j) * a.Hq + hq) * D + d4;
    if (a.o_f32) *reinterpret_cast<f32x4*>(a.o_f32 + off) = acc;
    if (a.o_bf16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) a.o_bf16[off + i] = f2bf(acc[i]);
    }
  }
}

__global__ void gather_slots_kernel(int B, int max_pages, int ps, int num_pages, const int32_t* pt,
                                    const int32_t* lens, int max_ctx_len, int32_t* slots, int* status) {
  const int b = blockIdx.y;
  int L = lens[b];
  int cap = max_pages * ps < max_ctx_len ? max_pages * ps : max_ctx_len;
  if (L < 0 || L > cap) {
    if (threadIdx.x == 0 && blockIdx.x == 0) set_status(status, ST_BAD_CTX_LEN);
    L = L < 0 ? 0 : cap;
  }
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < max_ctx_len; i += gridDim.x * blockDim.x) {
    int v = -1;
    if (i < L) {
      int pid = pt[(size_t)b * max_pages + i / ps];
      if (pid < 0 || pid >= num_pages) set_status(status, ST_BAD_PAGE);
      else v = pid * ps + i % ps;
    }
    slots[(size_t)b * max_ctx_len + i] = v;
  }
}

template <int D, int NW, bool LO>
hipError_t launch_sweep(const AttnArgs& a, hipStream_t s) {
  constexpr int lds = 2 * 2 * AttnCfg<D>::TILE * (LO ? 2 : 1);
  auto kern = attn_sweep<D, NW, LO>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3(a.max_splits, a.Hkv, a.B), dim3(64 * NW), lds, s, a);
  return hipGetLastError();
}

template <int D, bool LO>
hipError_t launch_sweep_nw(const AttnArgs& a, hipStream_t s) {
  const int R = a.T * (a.Hq / a.Hkv);
  const int nw = (R + 31) / 32;
  switch (nw) {
    case 1: return launch_sweep<D, 1, LO>(a, s);
    case 2: return launch_sweep<D, 2, LO>(a, s);
    case 3:
    case 4: return launch_sweep<D, 4, LO>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t attention_partials_bytes(int B, int Hkv, int max_splits, int R, int D) {
  const size_t units = (size_t)B * Hkv * max_splits;
  return units * R * D * sizeof(float) + units * R * 2 * sizeof(float);
}

int attention_default_split(int B, int Hkv, int max_ctx_len) {
  // Aim for ~2048 work units over the whole batch, in multiples of the 64-key tile.
  long long want = ((long long)max_ctx_len * B * Hkv + 2047) / 2048;
  long long s = ((want + KT - 1) / KT) * KT;
  if (s < 256) s = 256;
  long long cap = ((long long)(max_ctx_len > 0 ? max_ctx_len : 1) + KT - 1) / KT * KT;
  if (s > cap) s = cap;
  return (int)s;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const bool lo = a.q_lo != nullptr;
  hipError_t e;
  if (a.D == 128) e = lo ? launch_sweep_nw<128, true>(a, s) : launch_sweep_nw<128, false>(a, s);
  else if (a.D == 64) e = lo ? launch_sweep_nw<64, true>(a, s) : launch_sweep_nw<64, false>(a, s);
  else return hipErrorInvalidValue;
  if (e != hipSuccess) return e;
  if (a.max_splits > 1) {
    hipLaunchKernelGGL(attn_reduce, dim3(a.B * a.Hkv), dim3(256), 0, s, a);
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
