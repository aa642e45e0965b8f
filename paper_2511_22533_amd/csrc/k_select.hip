// Spatiotemporal Stability Criterion scoring and lowest-score selection
// (Sec. 4.2, Eqs. 2, 6, 7; Algorithm 1, SSC), one 1024-thread workgroup per
// sample.
//
// Phase 1 computes V_i = ||v_cache_i|| and A_i = ||v_cache_i - v_prev_i|| with
// a sequential float32 sum of squares (no fused multiply-add, correctly rounded
// sqrt) and reduces their per-sample min/max. Phase 2 forms the score
// C_i = w_a * norm(A_i) + w_v * norm(V_i) and an order-preserving 32-bit key
// (NaN -> largest). Phase 3 finds the key of rank c-1 by an exact 4 x 8-bit
// radix select over the keys held in LDS. Phase 4 scans the keys in token
// order: a token is cached if its key is smaller, or equal and among the first
// r equal keys, which reproduces a stable ascending sort truncated at c.
#include "common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace f3c {

namespace {

constexpr int kThreads = 1024;
constexpr int kPer = kMaxTokens / kThreads;   // tokens per thread in phase 1

__device__ __forceinline__ float sumsq8(const float4& a, const float4& b) {
  float s = 0.0f;
  s = __fadd_rn(s, __fmul_rn(a.x, a.x));
  s = __fadd_rn(s, __fmul_rn(a.y, a.y));
  s = __fadd_rn(s, __fmul_rn(a.z, a.z));
  s = __fadd_rn(s, __fmul_rn(a.w, a.w));
  s = __fadd_rn(s, __fmul_rn(b.x, b.x));
  s = __fadd_rn(s, __fmul_rn(b.y, b.y));
  s = __fadd_rn(s, __fmul_rn(b.z, b.z));
  s = __fadd_rn(s, __fmul_rn(b.w, b.w));
  return s;
}

__device__ __forceinline__ float4 sub4(const float4& a, const float4& b) {
  return make_float4(__fsub_rn(a.x, b.x), __fsub_rn(a.y, b.y), __fsub_rn(a.z, b.z), __fsub_rn(a.w, b.w));
}

__device__ __forceinline__ uint32_t order_key(float c) {
  if (c != c) return 0xFFFFFFFFu;
  if (c == 0.0f) c = 0.0f;                          // -0 orders with +0
  uint32_t u = __float_as_uint(c);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Correctly rounded float32 square root and quotient. (The library is built
// with -fhip-fp32-correctly-rounded-divide-sqrt; the __fsqrt_rn intrinsic maps to
// the approximate native instruction and is not used.)
__device__ __forceinline__ float sqrt_rn(float x) { return __builtin_sqrtf(x); }
__device__ __forceinline__ float div_rn(float a, float b) { return a / b; }

__device__ __forceinline__ float norm_term(float a, float lo, float hi) {
  if (!(hi > lo)) return 0.0f;
  return div_rn(__fsub_rn(a, lo), __fsub_rn(hi, lo));
}

// Exclusive block scan of one int per thread; returns the exclusive prefix and
// the block total. Uses the 16-entry scratch `ws`.
__device__ int block_exclusive_scan(int v, int* ws, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ws[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kThreads / 64 ? ws[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      int y = __shfl_up(w, o);
      if (lane >= o) w += y;
    }
    if (lane < kThreads / 64) ws[lane] = w;
  }
  __syncthreads();
  int before = (wave > 0 ? ws[wave - 1] : 0) + x - v;
  *total = ws[kThreads / 64 - 1];
  __syncthreads();
  return before;
}

__global__ __launch_bounds__(kThreads) void k_score_select(const float* __restrict__ v_cache,
                                                           const float* __restrict__ v_prev, int N, float w_a,
                                                           float w_v, Segs n_cache, Segs act,
                                                           int32_t* __restrict__ idx_active,
                                                           int32_t* __restrict__ pos, float* __restrict__ score) {
  __shared__ uint32_t keys[kMaxTokens];
  __shared__ float red[4][kThreads / 64];
  __shared__ int hist[256];
  __shared__ int scan_ws[kThreads / 64];
  __shared__ int sel[2];

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int c = n_cache.off[b];
  const int row0 = act.off[b];
  const size_t base = (size_t)b * N;

  if (c == 0) {  // full step for this sample: identity selection, no scoring
    for (int i = tid; i < N; i += kThreads) {
      idx_active[row0 + i] = i;
      pos[base + i] = row0 + i;
    }
    return;
  }

  // Phase 1: magnitudes and per-sample extremes (NaN ignored by fminf/fmaxf).
  float V[kPer], A[kPer];
  float loV = INFINITY, hiV = -INFINITY, loA = INFINITY, hiA = -INFINITY;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kThreads;
    V[j] = 0.0f;
    A[j] = 0.0f;
    if (i < N) {
      const float4* pc = reinterpret_cast<const float4*>(v_cache + (base + i) * 8);
      const float4* pp = reinterpret_cast<const float4*>(v_prev + (base + i) * 8);
      float4 c0 = pc[0], c1 = pc[1], p0 = pp[0], p1 = pp[1];
      V[j] = sqrt_rn(sumsq8(c0, c1));
      A[j] = sqrt_rn(sumsq8(sub4(c0, p0), sub4(c1, p1)));
      loV = fminf(loV, V[j]);
      hiV = fmaxf(hiV, V[j]);
      loA = fminf(loA, A[j]);
      hiA = fmaxf(hiA, A[j]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    loV = fminf(loV, __shfl_xor(loV, o));
    hiV = fmaxf(hiV, __shfl_xor(hiV, o));
    loA = fminf(loA, __shfl_xor(loA, o));
    hiA = fmaxf(hiA, __shfl_xor(hiA, o));
  }
  const int lane = tid & 63, wave = tid >> 6;
  if (lane == 0) {
    red[0][wave] = loV;
    red[1][wave] = hiV;
    red[2][wave] = loA;
    red[3][wave] = hiA;
  }
  __syncthreads();
  loV = red[0][0];
  hiV = red[1][0];
  loA = red[2][0];
  hiA = red[3][0];
  for (int w = 1; w < kThreads / 64; ++w) {
    loV = fminf(loV, red[0][w]);
    hiV = fmaxf(hiV, red[1][w]);
    loA = fminf(loA, red[2][w]);
    hiA = fmaxf(hiA, red[3][w]);
  }

  // Phase 2: scores and order keys.
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kThreads;
    if (i < N) {
      const float cs = __fadd_rn(__fmul_rn(w_a, norm_term(A[j], loA, hiA)),
                                 __fmul_rn(w_v, norm_term(V[j], loV, hiV)));
      keys[i] = order_key(cs);
      if (score) score[base + i] = cs;
    }
  }
  __syncthreads();

  // Phase 3: radix select of the key with 0-based rank c-1.
  uint32_t prefix = 0, mask = 0;
  int r = c;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kThreads) hist[i] = 0;
    __syncthreads();
    for (int i = tid; i < N; i += kThreads) {
      const uint32_t k = keys[i];
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
    }
    __syncthreads();
    if (wave == 0) {
      // lane owns bins 4*lane .. 4*lane+3
      int h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2], h3 = hist[4 * lane + 3];
      int tot = h0 + h1 + h2 + h3, x = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o);
        if (lane >= o) x += y;
      }
      int before = x - tot;
      if (before < r && r <= x) {
        int d = 4 * lane, cum = before;
        if (cum + h0 >= r) { d += 0; }
        else if (cum + h0 + h1 >= r) { d += 1; cum += h0; }
        else if (cum + h0 + h1 + h2 >= r) { d += 2; cum += h0 + h1; }
        else { d += 3; cum += h0 + h1 + h2; }
        sel[0] = d;
        sel[1] = r - cum;
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sel[0] << shift;
    mask |= 255u << shift;
    r = sel[1];
    __syncthreads();
  }
  const uint32_t kstar = prefix;   // key of rank c-1; r = cached tokens among keys == kstar

  // Phase 4: token-order scan. Thread t owns the contiguous range [t*P, t*P + P).
  const int P = (N + kThreads - 1) / kThreads;
  const int i0 = min(N, tid * P), i1 = min(N, i0 + P);
  int eq_local = 0;
  for (int i = i0; i < i1; ++i) eq_local += (keys[i] == kstar);
  int tot;
  int eq_before = block_exclusive_scan(eq_local, scan_ws, &tot);
  int act_local = 0;
  {
    int e = eq_before;
    for (int i = i0; i < i1; ++i) {
      const uint32_t k = keys[i];
      bool cached = k < kstar;
      if (k == kstar) { cached = e < r; ++e; }
      act_local += !cached;
    }
  }
  int act_before = block_exclusive_scan(act_local, scan_ws, &tot);
  {
    int e = eq_before, a = row0 + act_before;
    for (int i = i0; i < i1; ++i) {
      const uint32_t k = keys[i];
      bool cached = k < kstar;
      if (k == kstar) { cached = e < r; ++e; }
      if (cached) {
        pos[base + i] = -1;
      } else {
        pos[base + i] = a;
        idx_active[a] = i;
        ++a;
      }
    }
  }
}

// Teacher-forced selection: pos of every token is -1 ...
__global__ __launch_bounds__(256) void k_pos_fill(int32_t* __restrict__ pos, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) pos[i] = -1;
}

// ... then every listed row r of sample b sets idx_active[r] = i and
// pos[b][i] = r, with i clamped into [0, N) so that no access leaves the
// arrays whatever the caller's buffer holds.
__global__ __launch_bounds__(256) void k_force_scatter(const int32_t* __restrict__ idx_in, Segs act, int N,
                                                       int32_t* __restrict__ idx_out, int32_t* __restrict__ pos) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= act.off[act.B]) return;
  const int b = find_segment(act.off, act.B, r);
  const int i = min(max(idx_in[r], 0), N - 1);
  idx_out[r] = i;
  pos[(size_t)b * N + i] = r;
}

}  // namespace

hipError_t launch_force_active(const int32_t* idx_in, const Segs& act, int N, int32_t* idx_out, int32_t* pos,
                               hipStream_t s) {
  const int64_t n = (int64_t)act.B * N;
  launch(k_pos_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, pos, n);
  const int rows = act.off[act.B];
  if (rows > 0) launch(k_force_scatter, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, idx_in, act, N, idx_out, pos);
  return hipGetLastError();
}

hipError_t launch_select(const float* v_cache, const float* v_prev, int B, int N, float w_a, float w_v,
                         const Segs& n_cache, const Segs& act, int32_t* idx_active, int32_t* pos,
                         float* score, hipStream_t s) {
  launch(k_score_select, dim3(B), dim3(kThreads), 0, s, v_cache, v_prev, N, w_a, w_v, n_cache, act,
                     idx_active, pos, score);
  return hipGetLastError();
}

}  // namespace f3c
