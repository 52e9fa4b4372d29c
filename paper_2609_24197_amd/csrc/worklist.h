// Work list of the KV sweep, built on the device from the context lengths.  Shared by the
// work-list kernel of the attention calls and by the q/k-norm + RoPE launch, which builds it in
// one extra workgroup so that the list costs no launch of its own inside a drafting step.
#pragma once
#include <climits>

#include "common.h"
#include "kernels.h"

namespace hspec {

constexpr int MAX_SPLIT = kMaxSplit;   // keys per split (host-enforced by the config check)
constexpr int WL_THREADS = 256;   // threads of a workgroup that builds the list
constexpr int WL_NCAND = 64;      // split sizes tried under automatic splitting (one lane each)
static_assert(WL_NCAND <= 64 && (WL_NCAND & (WL_NCAND - 1)) == 0, "one lane of a wave per candidate size");

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

// First cache position a sweep reads for a request of length L.  Under a sliding window the
// query at position L + j sees cache positions p >= L + j - window + 1, so no query of the
// block sees p < L - window + 1; those positions are not read at all.
__device__ __forceinline__ int swept_lo(const AttnArgs& a, int L) {
  return a.window > 0 && L - a.window + 1 > 0 ? L - a.window + 1 : 0;
}

// Splits of one request.  The swept range [swept_lo, L) of n positions is cut into ns runs:
// every run but the last holds q positions (a whole number of 32-key tiles, at most MAX_SPLIT),
// the last one the rest, and ns = ceil(n / q), so no run is empty.  n = 0 is one split with no
// cache keys.  The work-list kernel picks (ns, q) per request and stores them; the sweep and
// the reductions read them back, so all three cut a request the same way.
__device__ __forceinline__ int swept_n(const AttnArgs& a, int L) { return L - swept_lo(a, L); }

// Split length for at most `ns` splits of n positions: ceil(n / ns) rounded up to a whole tile.
__device__ __forceinline__ int split_len_for(int n, int ns) {
  return n > 0 ? ((n + ns - 1) / ns + 31) & ~31 : 0;
}

// ceil(n / s) for 0 <= n < 2^24 and s >= 1: a float estimate, then corrected to the exact
// value (the estimate is off by at most one; an integer division costs several times more,
// and the split-size choice takes one per candidate size and request).
__device__ __forceinline__ int ceil_div_est(int n, int s) {
  int q = (int)((float)n * __builtin_amdgcn_rcpf((float)s));
  while (q * s < n) ++q;
  while (q > 0 && (q - 1) * s >= n) --q;
  return q;
}

// Splits of a request of n swept positions when splits may hold up to S positions (n is at
// most 256 x MAX_SPLIT: host-enforced).
__device__ __forceinline__ int plan_pieces(int n, int S, int cap) {
  if (n <= 0) return 1;
  const int ns = max(ceil_div_est(n, S), (n + MAX_SPLIT - 1) / MAX_SPLIT);
  return max(1, min(ns, cap));
}

// Inclusive prefix sum over the workgroup (WL_THREADS lanes); total in *total.
__device__ __forceinline__ int plan_scan(int v, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  __syncthreads();   // s_wave free from the previous scan
  if (lane == 63) s_wave[w] = v;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < WL_THREADS / 64; ++i) {
    before += i < w ? s_wave[i] : 0;
    all += s_wave[i];
  }
  *total = all;
  return v + before;
}

// LDS of the builder: per-request arrays for up to RANK_MAX ranked requests.
template <int RANK_MAX>
struct WorklistLds {
  int n[RANK_MAX];      // swept positions of request b
  int rank[RANK_MAX];   // its rank, by split length
  int off[RANK_MAX];    // splits of the request at rank r, then its first item
  int wave[WL_THREADS / 64];
  int cnt[WL_NCAND];
  int sum, max, choice;
};

// Work list of the sweep: every (request, split) once, as (request << 16 | split, context
// length, split length, splits of the request), requests ordered by decreasing split length (all
// splits of a request together), so that the persistent workgroups, taking items longest first,
// finish close together.  One workgroup of WL_THREADS threads.
//
// Split size.  An explicit split size (split_tokens) is used as given.  With the automatic size
// (auto_split) the work list picks it from the actual lengths, among WL_NCAND sizes from twice
// the host's size (at most MAX_SPLIT) down to min_split: the largest size that gives every persistent
// workgroup one item of at most 1/16 above the average work, else the size whose item count
// comes closest below a whole number (two or more) of rounds of the `grid` workgroups, so that
// the last round of the queue is not left half empty.  Every request is then cut into the
// fewest near-equal runs of at most that size (at most max_splits, at most MAX_SPLIT keys).
// Requests are ranked by split length (ties by index) and their splits placed by a block-wide
// prefix sum over the ranks; beyond RANK_MAX requests they keep their own order.  Also
// resets the item queue and, as the first kernel of a call, its status words.
template <int RANK_MAX>
__device__ void build_worklist(const AttnArgs& a, int clear_words, WorklistLds<RANK_MAX>& lds) {
  int* s_n = lds.n;
  int* s_rank = lds.rank;
  int* s_off = lds.off;
  int* s_wave = lds.wave;
  int* s_cnt = lds.cnt;
  int& s_sum = lds.sum;
  int& s_max = lds.max;
  const int tid = threadIdx.x;
  if (tid < clear_words) a.status[tid] = 0;   // a call's first kernel clears its status words
  if (tid < WL_NCAND) s_cnt[tid] = 0;
  if (tid == 0) s_sum = s_max = 0;
  __syncthreads();
  const bool ranked = a.B <= RANK_MAX;
  const int cap = max(1, a.max_splits);

  // candidate split sizes: twice the host's size down to min_split in WL_NCAND near-even steps
  auto cand = [&](int c) {
    const int hi = min(MAX_SPLIT, 2 * a.split) / 32, lo = max(1, a.min_split / 32);
    return 32 * (hi - (hi - lo) * c / (WL_NCAND - 1));
  };
  int S = a.split;
  if (ranked) {
    int sum = 0, mx = 0;
    for (int b = tid; b < a.B; b += WL_THREADS) {
      const int n = swept_n(a, clamp_len(a, b));
      s_n[b] = n;
      sum += n;
      mx = max(mx, n);
    }
    if (a.auto_split && a.grid > 0) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        sum += __shfl_xor(sum, o);
        mx = max(mx, __shfl_xor(mx, o));
      }
      if ((tid & 63) == 0) {
        atomicAdd(&s_sum, sum);
        atomicMax(&s_max, mx);
      }
      __syncthreads();
      // splits at each candidate size: lane l of every wave counts candidate l over the
      // requests b = w, w + 4, ... of its wave w; the four partial counts meet in LDS
      const int wv = tid >> 6, ln = tid & 63;
      if (ln < WL_NCAND) {
        const int Sc = cand(ln);
        int cnt = 0;
        for (int b = wv; b < a.B; b += WL_THREADS / 64) cnt += plan_pieces(s_n[b], Sc, cap);
        atomicAdd(&s_cnt[ln], cnt);
      }
      __syncthreads();
      // Choice, one lane per candidate: the largest size (smallest c) whose items fit one round
      // with the longest split within 1/16 of the average work per workgroup; else the size
      // leaving the fewest idle slots in the last of two or more rounds (larger size on ties).
      // (Item counts fit in 32 bits: the host bounds B x max_splits x Hkv.)
      if (tid < 64) {
        int key = INT_MAX;
        if (tid < WL_NCAND) {
          const long long avg = (long long)s_sum * a.Hkv;   // positions of all items; per workgroup: / grid
          const int items = s_cnt[tid] * a.Hkv;
          const int longest = min(cand(tid), s_max);
          if (items <= a.grid) {
            if ((long long)longest * a.grid * 16 <= avg * 17) key = tid;
          } else {
            const int rem = items % a.grid;
            key = (1 << 24) + (rem ? a.grid - rem : 0) * WL_NCAND + tid;
          }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) key = min(key, __shfl_xor(key, o));
        if (tid == 0) lds.choice = key;
      }
      __syncthreads();
      if (lds.choice != INT_MAX) S = cand(lds.choice & (WL_NCAND - 1));
    } else {
      __syncthreads();
    }
  }
  if (ranked) {
    // split length of each request, then its rank by split length (longest first)
    for (int b = tid; b < a.B; b += WL_THREADS) s_off[b] = split_len_for(s_n[b], plan_pieces(s_n[b], S, cap));
    __syncthreads();
    for (int b = tid; b < a.B; b += WL_THREADS) {
      const int key = s_off[b];
      int rank = 0;
#pragma unroll 8
      for (int o = 0; o < a.B; ++o) {
        const int ko = s_off[o];
        rank += (ko > key) || (ko == key && o < b);
      }
      s_rank[b] = rank;
    }
    __syncthreads();
    for (int b = tid; b < a.B; b += WL_THREADS) {
      const int q = split_len_for(s_n[b], plan_pieces(s_n[b], S, cap));
      s_off[s_rank[b]] = q > 0 ? (s_n[b] + q - 1) / q : 1;
    }
    __syncthreads();
  }
  // exclusive prefix sum of the split counts, in rank order (request order past RANK_MAX),
  // WL_THREADS entries at a time
  int base = 0;
  for (int r0 = 0; r0 < a.B; r0 += WL_THREADS) {
    const int r = r0 + tid;
    int cnt = 0, L = 0, q = 0;
    if (r < a.B) {
      if (ranked) {
        cnt = s_off[r];
      } else {
        L = clamp_len(a, r);
        const int n = swept_n(a, L);
        q = split_len_for(n, plan_pieces(n, S, cap));
        cnt = q > 0 ? (n + q - 1) / q : 1;
      }
    }
    int total = 0;
    const int first = base + plan_scan(cnt, s_wave, &total) - cnt;
    if (r < a.B) {
      if (ranked) {
        s_off[r] = first;
      } else {
        for (int sp = 0; sp < cnt; ++sp)
          *reinterpret_cast<int4*>(a.units + 4 * (first + sp)) = int4{(r << 16) | sp, L, q, cnt};
        *reinterpret_cast<int2*>(a.req + 2 * r) = int2{cnt, q};
      }
    }
    base += total;
  }
  __syncthreads();
  if (ranked) {
    for (int b = tid; b < a.B; b += WL_THREADS) {
      const int L = clamp_len(a, b);
      const int q = split_len_for(s_n[b], plan_pieces(s_n[b], S, cap));
      const int ns = q > 0 ? (s_n[b] + q - 1) / q : 1;
      const int first = s_off[s_rank[b]];
      for (int sp = 0; sp < ns; ++sp)
        *reinterpret_cast<int4*>(a.units + 4 * (first + sp)) = int4{(b << 16) | sp, L, q, ns};
      *reinterpret_cast<int2*>(a.req + 2 * b) = int2{ns, q};
    }
  }
  if (tid == 0) {
    a.status[1] = base * a.Hkv;
    a.status[2] = 0;
  }
}

}  // namespace hspec
