// Draft head: the Markov correction of the block's logits and the choice of draft tokens
// (Sec. 3.3.3 causal correction; App. B.1 "Markov rank"; App. B.2 "Pruned drafter vocabulary").
//
// Position j of request b gets the logits of the LM head plus a rank-R term picked by the token
// chosen at position j - 1:
//   l'[b, j, v] = base[b, j, v] + sum_r E[t_{b, j-1}, r] U[v, r],   t_{b, -1} = prev[b],
// and its token is the argmax over v of l' (greedy) or of l' / T + G (Gumbel-max sampling with
// the caller's noise G).  The chain is sequential in j, so each position is one launch:
//   * a workgroup owns 128 vocabulary columns and all requests (in tiles of 64);
//   * the rank-R product is one MFMA tile per (16 requests, 16 columns); the E rows of the
//     previous tokens are gathered into LDS once per workgroup, the U rows of a wave's columns
//     read from L2;
//   * the argmax across workgroups is a 64-bit atomicMax on (orderable score << 32 | ~column),
//     which picks the largest score and, among equal scores, the lowest column;
//   * the next launch decodes the previous position's token from that key.
#include "common.h"
#include "kernels.h"

namespace hspec {
namespace {

constexpr int MK_COLS = 128;   // vocabulary columns per workgroup (4 waves x 2 MFMA column blocks)
constexpr int MK_ROWS = 64;    // requests per tile (4 MFMA row blocks)
constexpr int ST_BAD_TOKEN = 4;
constexpr int ST_NONFINITE = 8;

// Order-preserving map of a float to uint32 (larger float, larger key); NaN is mapped as -inf.
__device__ __forceinline__ unsigned long long score_key(float s, int col) {
  unsigned u = __float_as_uint(s);
  const unsigned ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)ord << 32) | (0xffffffffu - (unsigned)col);
}
__device__ __forceinline__ int key_token(unsigned long long key) {
  return (int)(0xffffffffu - (unsigned)(key & 0xffffffffu));
}
__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int m) {
  const unsigned lo = __shfl_xor((unsigned)(v & 0xffffffffu), m);
  const unsigned hi = __shfl_xor((unsigned)(v >> 32), m);
  return ((unsigned long long)hi << 32) | lo;
}

// RK: rank / 32 when known at compile time (the request tile's E rows gathered once per
// workgroup into LDS, every fragment load issued before the first MFMA), 0 for any rank that is
// a multiple of 32 (E and U fragments read from L2, one round of loads per 32).
template <int RK>
__global__ void __launch_bounds__(256) markov_step_kernel(HeadArgs a, int j) {
  constexpr int RR = RK * 32, LDE = RR + 8;   // E rows in LDS, padded by 16 bytes
  __shared__ int s_prev[MK_ROWS];
  __shared__ unsigned long long s_best[4][MK_ROWS];
  __shared__ __align__(16) bf16 s_e[RK > 0 ? MK_ROWS * LDE : 8];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int vw = blockIdx.x * MK_COLS + wave * 32;   // first column of this wave
  const int l16 = lane & 15, g4 = lane >> 4;
  // the next position's keys start at zero; they are first updated by the next launch
  if (blockIdx.x == 0 && j + 1 < a.k)
    for (int b = tid; b < a.B; b += 256) a.keys[(size_t)b * a.k + j + 1] = 0;

  for (int b0 = 0; b0 < a.B; b0 += MK_ROWS) {
    if (tid < MK_ROWS) {
      const int b = b0 + tid;
      int t = 0;
      if (b < a.B) {
        if (j == 0) t = a.prev[b];
        else if (a.forced) t = a.forced[(size_t)b * a.k + j - 1];
        else t = key_token(a.keys[(size_t)b * a.k + j - 1]);
        if (t < 0 || t >= a.V) {
          if (blockIdx.x == 0) set_status(a.status, ST_BAD_TOKEN);
          t = 0;
        }
      }
      s_prev[tid] = t;
    }
    __syncthreads();

    // this tile's LM-head logits, loaded while the rank product runs
    float base[4][4][2];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          const int b = b0 + rb * 16 + 4 * g4 + i, col = vw + cb * 16 + l16;
          base[rb][i][cb] = (b < a.B && col < a.V) ? a.base[((size_t)b * a.k + j) * a.V + col] : 0.f;
        }

    // adj[b][v] = E[prev_b] . U[v] over the rank
    f32x4 acc[4][2];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16* urow[2];
    bool ucol[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const int col = vw + cb * 16 + l16;
      ucol[cb] = col < a.V;
      urow[cb] = a.U + (size_t)(ucol[cb] ? col : 0) * a.R + 8 * g4;
    }
    const bf16* erow[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) erow[rb] = a.E + (size_t)s_prev[rb * 16 + l16] * a.R + 8 * g4;
    auto rank_steps = [&](int ks0, auto nsteps) {
      constexpr int NS = decltype(nsteps)::value;
      bf16x8 ef[NS][4], uf[NS][2];
#pragma unroll
      for (int s = 0; s < NS; ++s) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) ef[s][rb] = ld8(erow[rb] + ks0 + 32 * s);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) uf[s][cb] = ucol[cb] ? ld8(urow[cb] + ks0 + 32 * s) : zero8();
      }
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = mma16(ef[s][rb], uf[s][cb], acc[rb][cb]);
    };
    if constexpr (RK > 0) {
      // the tile's E rows are gathered once per workgroup into LDS; the four waves read their
      // fragments from there
      constexpr int CPR = RR / 8;                    // 16-byte chunks per E row
      static_assert((MK_ROWS * CPR) % 256 == 0, "E tile chunks must divide over the workgroup");
      bf16x8 uf[RK][2];
#pragma unroll
      for (int s = 0; s < RK; ++s)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) uf[s][cb] = ucol[cb] ? ld8(urow[cb] + 32 * s) : zero8();
#pragma unroll
      for (int q = 0; q < MK_ROWS * CPR / 256; ++q) {
        const int c = tid + 256 * q, row = c / CPR, col = (c % CPR) * 8;
        *reinterpret_cast<bf16x8*>(s_e + row * LDE + col) = ld8(a.E + (size_t)s_prev[row] * RR + col);
      }
      __syncthreads();
      bf16x8 ef[RK][4];
#pragma unroll
      for (int s = 0; s < RK; ++s)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
          ef[s][rb] = *reinterpret_cast<const bf16x8*>(s_e + (rb * 16 + l16) * LDE + 32 * s + 8 * g4);
#pragma unroll
      for (int s = 0; s < RK; ++s)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = mma16(ef[s][rb], uf[s][cb], acc[rb][cb]);
    } else {
      for (int ks = 0; ks < a.R; ks += 32) rank_steps(ks, Int<1>{});
    }

    // corrected logits, scores, and the best (score, column) of each request in this wave
    bool bad = false;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = rb * 16 + 4 * g4 + i;
        const int b = b0 + r;
        unsigned long long best = 0;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          const int col = vw + cb * 16 + l16;
          if (b < a.B && col < a.V) {
            const size_t off = ((size_t)b * a.k + j) * a.V + col;
            const float l = base[rb][i][cb] + acc[rb][cb][i];
            if (a.logits) a.logits[off] = l;
            float sc = a.gumbel ? l * a.inv_temp + a.gumbel[off] : l;
            if (!(sc == sc)) {
              bad = true;
              sc = -INFINITY;
            }
            const unsigned long long key = score_key(sc, col);
            best = key > best ? key : best;
          }
        }
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) {
          const unsigned long long o = shfl_xor_u64(best, m);
          best = o > best ? o : best;
        }
        if (l16 == 0) s_best[wave][r] = best;
      }
    if (bad) set_status(a.status, ST_NONFINITE);
    __syncthreads();
    if (tid < MK_ROWS && b0 + tid < a.B) {
      unsigned long long best = s_best[0][tid];
#pragma unroll
      for (int w = 1; w < 4; ++w) best = s_best[w][tid] > best ? s_best[w][tid] : best;
      if (best) atomicMax(a.keys + (size_t)(b0 + tid) * a.k + j, best);
    }
    __syncthreads();   // s_prev and s_best are reused by the next request tile
  }
}

// The call's first kernel: status words and the keys of position 0.
__global__ void head_clear_kernel(int* status, int nwords, unsigned long long* keys, int B, int k) {
  for (int i = threadIdx.x; i < nwords; i += blockDim.x) status[i] = 0;
  for (int b = threadIdx.x; b < B; b += blockDim.x) keys[(size_t)b * k] = 0;
}

__global__ void head_tokens_kernel(const unsigned long long* keys, int n, int32_t* tokens) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) tokens[i] = key_token(keys[i]);
}

}  // namespace

hipError_t launch_markov_head(const HeadArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.k <= 0) return hipSuccess;
  const int n = a.B * a.k;
  const int grid = (a.V + MK_COLS - 1) / MK_COLS;
  auto kern = a.R == 256 ? markov_step_kernel<8> : markov_step_kernel<0>;
  for (int j = 0; j < a.k; ++j) {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, s, a, j);
    if (hipError_t e = hipGetLastError()) return e;
  }
  hipLaunchKernelGGL(head_tokens_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a.keys, n, a.tokens);
  return hipGetLastError();
}

hipError_t launch_head_clear(const HeadArgs& a, int status_words, hipStream_t s) {
  hipLaunchKernelGGL(head_clear_kernel, dim3(1), dim3(256), 0, s, a.status, status_words, a.keys, a.B, a.k);
  return hipGetLastError();
}

}  // namespace hspec
