// Internal launchers of the HIP kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "hspec.h"

namespace hspec {

typedef __bf16 bf16;

// C[M,N] = A[M,K] * W[N,K]^T (+ R), fp32 accumulate.  *_lo planes are optional.
struct GemmArgs {
  const bf16* A_hi = nullptr; const bf16* A_lo = nullptr; int lda = 0;
  const bf16* W_hi = nullptr; const bf16* W_lo = nullptr; int ldw = 0;
  int M = 0, N = 0, K = 0;
  float* C = nullptr; int ldc = 0;             // fp32 result (optional)
  const void* R = nullptr; int ldr = 0; int r_bf16 = 0;   // residual added (optional)
  bf16* C_hi = nullptr; bf16* C_lo = nullptr; int ldch = 0;  // bf16 planes of the result
  _Float16* C_h16 = nullptr;   // fp16 copy of h16_scale x result, leading dimension ldch (weight-streaming path only)
  _Float16* C_l16 = nullptr;   // with C_h16: the fp16 residual h16_scale x result - C_h16, or null
  float h16_scale = 1.f;       // (a power of two)
  float out_scale = 1.f;       // the product is multiplied by this (a power of two) before any output
  int f16 = 0;                 // A planes and the packed W hold fp16 values (packed W only)
  float* part = nullptr; size_t part_cap = 0;  // split-K scratch (fp32 elements), optional
  int w_packed = 0;   // W_hi is in the fragment-major packed layout (launch_pack_w, fp16 W x 2^kPackScaleLog2)
  // Optional row segments of W (bf16, not packed): rows [0, N1) come from W_hi, [N1, N1 + N2)
  // from W2 and [N1 + N2, N) from W3, each with leading dimension ldw.
  const bf16* W2 = nullptr; const bf16* W3 = nullptr; int N1 = 0, N2 = 0;
};
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);
// Whether launch_gemm takes an M x N x K product (bf16 W) on the weight-streaming path, the only
// one that writes C_h16.
bool gemm_f16_out_ok(int M, int N, int K);
// fp32 elements of split-K scratch that launch_gemm uses for an M x N x K product when
// given at least that much (0: the shape is never split).
size_t gemm_scratch_elems(int M, int N, int K, bool a_lo, bool w_lo);
// Rewrites a row-major bf16 W[N, K] (N % 16 == 0, K % 32 == 0) into the packed layout that
// launch_gemm streams when w_packed is set: 1 KB blocks (k-step s, 16-row tile t) at
// ((s * N/16) + t) * 1024 bytes, each one 16x32 MFMA operand fragment, holding the fp16 values of
// W x 2^kPackScaleLog2 (exact for every bf16 W of magnitude 2^-25 .. 2^7).  The product with a
// packed W is an fp16 product (f16 set, A as fp16 planes); out_scale takes the factor back.
constexpr int kPackScaleLog2 = 8;
hipError_t launch_pack_w(const bf16* W, int N, int K, _Float16* Wp, hipStream_t s);

// Paged block attention (split-K sweep over the target cache + block keys, then reduce).
struct AttnArgs {
  const bf16 *q_hi = nullptr, *q_lo = nullptr;        // [B, T, Hq, D] post-RoPE
  const bf16 *kb_hi = nullptr, *kb_lo = nullptr;      // [B, T, Hkv, D] post-RoPE
  const bf16 *vb_hi = nullptr, *vb_lo = nullptr;
  const bf16 *kc_hi = nullptr, *kc_lo = nullptr;      // [num_pages, ps, Hkv, D]
  const bf16 *vc_hi = nullptr, *vc_lo = nullptr;
  const int32_t* page_table = nullptr;                // [B, max_pages]
  const int32_t* ctx_lens = nullptr;                  // [B]
  int B = 0, T = 0, Hq = 0, Hkv = 0, D = 0, ps = 0, max_pages = 0, num_pages = 0;
  int window = 0, causal = 0, max_ctx_len = 0, split = 0, max_splits = 0;
  int Hkv_cache = 0;                  // KV heads per slot of the cache (>= Hkv)
  int kv_remap = 0;                   // 1: drafter KV head h reads cache head kv_map[4h .. 4h+3], else h
  unsigned long long kv_map = 0;
  int block_in_sweep = 1;     // 1: the sweep takes the block keys (bf16); 0: the reduction, in fp32
  float scale_log2 = 0.f;
  float* part_o = nullptr;    // [B*Hkv*max_splits, R, D]
  float* part_ml = nullptr;   // [B*Hkv*max_splits, R, 2]
  float* o_f32 = nullptr;     // [B, T, Hq, D] (one of o_f32 / o_bf16)
  bf16* o_bf16 = nullptr;
  bf16* o_bf16_lo = nullptr;  // with o_bf16: the lo plane of o, or null
  int* status = nullptr;      // device status word; status[1] = work items, status[2] = queue (zero at launch)
  int32_t* units = nullptr;   // [B * max_splits][4] work list (request << 16 | split, length, split length, splits)
  int32_t* req = nullptr;     // [B][2] splits of each request and their length (written by the work list)
  int grid = 0;               // persistent workgroups of the sweep (attention_sweep_grid)
  int auto_split = 0;         // 1: the work list picks the split size in [min_split, split] from the lengths
  int min_split = 0;
};
// Persistent workgroups the KV sweep runs with on the current device (head dim D, R = k g
// query rows per KV head, lo: fp32 storage); 0 if the shape has no sweep variant.
int attention_sweep_grid(int D, int R, bool lo);
// Work list of the sweep (reads only B, ctx_lens, split and the table sizes of a); clears
// status[0, clear_words) first.  Must precede launch_attention on the stream.
hipError_t launch_attention_plan(const AttnArgs& a, int clear_words, hipStream_t s);
enum : unsigned { ATTN_SWEEP = 1u, ATTN_REDUCE = 2u };   // parts of launch_attention
hipError_t launch_attention(const AttnArgs& a, hipStream_t s, unsigned parts = ATTN_SWEEP | ATTN_REDUCE);
size_t attention_partials_bytes(int B, int Hkv, int max_splits, int R, int D);
constexpr int kStatusWords = 64;   // int32 words reserved at the start of every workspace
constexpr int kStatusClear = 4;    // cleared at the start of every call: status bits, work items, queue
constexpr int kWorklistFusedMax = 512;   // requests up to which the work list rides in the RoPE launch
constexpr int kMaxSplit = 8192;          // cache keys per split (one split's page ids sit in LDS)
// Split size (keys, multiple of 64) when the caller leaves it to the library: about 1024
// (request, split, head) items over the longest requests, enough to fill every resident
// workgroup slot, few enough that split partials and item start-up stay small; at most
// kMaxSplit, and never more than 256 splits per request.
inline int attention_default_split(int B, int Hkv, int swept_len) {
  const long long want = ((long long)swept_len * B * Hkv + 1023) / 1024;
  long long s = (want + 63) / 64 * 64;
  if (s < 256) s = 256;
  const long long cap = ((long long)(swept_len > 0 ? swept_len : 1) + 63) / 64 * 64;
  if (s > cap) s = cap;
  if (s > kMaxSplit) s = kMaxSplit;
  const long long min_for_256 = ((long long)swept_len + 255) / 256;
  if (s < min_for_256) s = (min_for_256 + 63) / 64 * 64;
  return (int)s;
}
// Smallest split size the work-list kernel may choose under automatic splitting: two thirds
// of the host's size, and never more than 256 splits.
inline int attention_min_auto_split(int host_split, int swept_len) {
  long long s = ((long long)host_split * 2 / 3 + 63) / 64 * 64;
  const long long min_for_256 = ((long long)swept_len + 255) / 256;
  if (s < min_for_256) s = (min_for_256 + 63) / 64 * 64;
  if (s < 64) s = 64;
  return (int)(s < host_split ? s : host_split);
}
// Longest run of cache positions the sweep reads for one request: max_ctx_len, or window - 1
// under a sliding window (no query of the block sees an older position).
inline int attention_swept_len(int max_ctx_len, int window) {
  return window > 0 && window - 1 < max_ctx_len ? window - 1 : max_ctx_len;
}

hipError_t launch_gather_slots(int B, int max_pages, int ps, int num_pages, const int32_t* page_table,
                               const int32_t* ctx_lens, int max_ctx_len, int32_t* slots, int* status,
                               hipStream_t s);

// Chunked SSD scan from an injected state.
struct ScanArgs {
  const bf16 *x_hi = nullptr, *x_lo = nullptr;        // [B, T, H, P]
  const float* dt = nullptr;                          // [B, T, H] (post-softplus)
  const float* A = nullptr;                           // [H]: A, or A_log when A_is_log
  int A_is_log = 0;                                   // A_h = -exp(A_log[h])
  const bf16 *B_hi = nullptr, *B_lo = nullptr;        // [B, T, G, N]
  const bf16 *C_hi = nullptr, *C_lo = nullptr;
  const float* Dskip = nullptr;                       // [H]
  const bf16 *S0_hi = nullptr, *S0_lo = nullptr;      // [B, H, P, N] or null
  const _Float16* S0_h16 = nullptr;                    // [B, H, P, N] as one fp16 plane (instead of S0_hi/lo)
  float* y = nullptr;                                 // [B, T, H, P]
  float* S_final = nullptr;                           // [B, H, P, N] or null
  int B = 0, T = 0, H = 0, P = 0, N = 0, G = 0, chunk = 0;
  int x_ld = 0;      // elements between consecutive tokens of x (>= H*P)
  int bc_ld = 0;     // elements between consecutive tokens of B and C (>= G*N)
  int dt_ld = 0;     // elements between consecutive tokens of dt (>= H)
};
hipError_t launch_ssd_scan(const ScanArgs& a, hipStream_t s);

// Elementwise / normalisation kernels.
// out = x / sqrt(mean(x^2) + eps) * w, rows of n; x is fp32 or bf16; outputs bf16 hi/lo planes.
hipError_t launch_rmsnorm_planes(const void* x, int x_bf16, const float* w, int rows, int n, float eps,
                                 bf16* out_hi, bf16* out_lo, hipStream_t s);
// Depthwise causal conv (zero left state) + SiLU over the xBC slice of zxbcdt, split into
// x (bf16 planes) and B, C (bf16 planes); dt = softplus(dt_raw + dt_bias).
struct ConvArgs {
  const float* zxbcdt = nullptr;    // [B*T, d_in_proj]
  const void* conv_w = nullptr;     // [conv_dim, K] storage dtype
  const void* conv_b = nullptr;     // [conv_dim]
  int w_bf16 = 1;
  const float* dt_bias = nullptr;   // [H]
  int B = 0, T = 0, H = 0, P = 0, G = 0, N = 0, K = 0;
  bf16 *x_hi = nullptr, *x_lo = nullptr;   // [B*T, H*P]
  bf16 *B_hi = nullptr, *B_lo = nullptr;   // [B*T, G*N]
  bf16 *C_hi = nullptr, *C_lo = nullptr;
  float* dt = nullptr;                     // [B*T, H]
};
hipError_t launch_conv_split(const ConvArgs& a, hipStream_t s);
// yn = RMSNorm_group(y * SiLU(z)) * w -> bf16 planes.  z rows have stride z_ld.
hipError_t launch_gated_rmsnorm(const float* y, const float* z, int z_ld, const float* w, int rows,
                                int n, int G, float eps, bf16* out_hi, bf16* out_lo, hipStream_t s);
// q/k per-head RMSNorm + RoPE at position ctx_len + j; v copied.  qkv rows [Hq*D | Hkv*D | Hkv*D].
// With `plan` (at most kWorklistFusedMax requests) one extra workgroup also builds the sweep's
// work list for those attention arguments, clearing the first plan_clear status words, as
// launch_attention_plan does.
hipError_t launch_qk_norm_rope(const float* qkv, const float* qw, const float* kw, const int32_t* ctx_lens,
                               int B, int T, int Hq, int Hkv, int D, float eps, double theta,
                               bf16* q_hi, bf16* q_lo, bf16* k_hi, bf16* k_lo, bf16* v_hi, bf16* v_lo,
                               hipStream_t s, const AttnArgs* plan = nullptr, int plan_clear = 0);
// fp32 -> bf16 hi/lo planes (lo optional).
hipError_t launch_split_planes(const float* x, size_t n, bf16* hi, bf16* lo, hipStream_t s);
// SwiGLU: h = SiLU(gate) * up from rows [gate | up] (fp32, width 2 ff) -> bf16 planes [rows, ff].
hipError_t launch_silu_mul(const float* gu, int rows, int ff, bf16* hi, bf16* lo, hipStream_t s);
// Appends K/V rows [B*n, Hkv*D] (bf16 planes, lo optional) at slot(ctx_len + i) of a paged cache
// (bf16 or fp32 storage); unmapped positions set status bit 2, bad page ids bit 1.
hipError_t launch_kv_append(const bf16* k_hi, const bf16* k_lo, const bf16* v_hi, const bf16* v_lo, int B, int n,
                            int Hkv, int D, const int32_t* page_table, int max_pages, int num_pages, int ps,
                            const int32_t* ctx_lens, void* k_cache, void* v_cache, int cache_bf16, int* status,
                            hipStream_t s);
// Zero n int32 words (device status, counters) with a kernel, graph-capture safe.
hipError_t launch_zero_words(int* p, int n, hipStream_t s);

// Markov correction and token choice of the draft head (one launch per block position).
struct HeadArgs {
  int B = 0, k = 0, V = 0, R = 0;
  const bf16* E = nullptr;            // [V, R] rank-R code of the preceding token
  const bf16* U = nullptr;            // [V, R] rank-R output factor
  const float* base = nullptr;        // [B*k, V] LM-head logits
  float* logits = nullptr;            // [B*k, V] corrected logits, or null (may equal base)
  const float* gumbel = nullptr;      // [B*k, V] sampling noise, or null (greedy)
  float inv_temp = 1.f;               // 1 / temperature, with gumbel
  const int32_t* prev = nullptr;      // [B] last committed token
  const int32_t* forced = nullptr;    // [B, k] tokens used as t_{j-1} instead of the chosen ones, or null
  unsigned long long* keys = nullptr; // [B*k] argmax keys (workspace)
  int32_t* tokens = nullptr;          // [B*k] out
  int* status = nullptr;
};
// Clears the status words and the keys of position 0: the first kernel of a head call.
hipError_t launch_head_clear(const HeadArgs& a, int status_words, hipStream_t s);
// One Markov-correction launch per block position (each clears the next position's keys),
// then the tokens.
hipError_t launch_markov_head(const HeadArgs& a, hipStream_t s);

// Host side of the ABI: records msg as this thread's last error (hspec_last_error) and returns s.
hspec_status api_fail(hspec_status s, const char* msg);

}  // namespace hspec
