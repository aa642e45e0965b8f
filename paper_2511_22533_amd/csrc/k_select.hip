// Spatiotemporal Stability Criterion scoring and lowest-score selection
// (Sec. 4.2, Eqs. 2, 6, 7; Algorithm 1, SSC) in two kernels.
//
// k_score_stats streams the two velocity caches over the whole chip (one
// 256-thread workgroup per 1024 tokens of a sample): V_i = ||v_cache_i|| and
// A_i = ||v_cache_i - v_prev_i|| with a sequential float32 sum of squares (no
// fused multiply-add, correctly rounded sqrt), written as (V_i, A_i) pairs,
// and each workgroup's min/max of both. min/max are exact and order-free
// (the magnitudes are never -0; NaN is ignored), so the per-sample extremes do
// not depend on how the tokens are split.
//
// k_select runs one 1024-thread workgroup per sample: it reduces the partial
// extremes, forms the score C_i = w_a * norm(A_i) + w_v * norm(V_i) and an
// order-preserving 32-bit key (NaN -> largest) per token into LDS, finds the
// key of rank c-1 by an exact 4 x 8-bit radix select, and scans the keys in
// token order: a token is cached if its key is smaller, or equal and among the
// first r equal keys, which reproduces a stable ascending sort truncated at c.
#include <mutex>
#include <vector>

#include "common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace f3c {

namespace {

constexpr int kThreads = 1024;       // select: one workgroup per sample
constexpr int kStatThreads = 256;    // score statistics: tokens streamed over the chip
constexpr int kStatPer = 4;
constexpr int kChunk = kStatThreads * kStatPer;
constexpr int kMaxChunks = kMaxTokens / kChunk;
static_assert(kMaxChunks <= 64, "the select kernel reduces the partial extremes in one wave");

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

// In-place exclusive prefix sum of v[0..n) (n <= 512) by wave 0: lane l
// sums entries 8l .. 8l+7, the lanes scan their totals, then each lane
// writes its entries' exclusive prefixes. Callers place barriers around it.
__device__ void segment_exclusive_scan(int* v, int n, int lane, int wave) {
  if (wave != 0) return;
  int loc[8];
  int sum = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = 8 * lane + e;
    loc[e] = k < n ? v[k] : 0;
    sum += loc[e];
  }
  int x = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  int run = x - sum;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = 8 * lane + e;
    if (k < n) v[k] = run;
    run += loc[e];
  }
}

// (V_i, A_i) of every token of the samples with c_b > 0, and each
// workgroup's extremes (loV, hiV, loA, hiA) at partial[b * chunks + chunk].
__global__ __launch_bounds__(kStatThreads) void k_score_stats(const float* __restrict__ v_cache,
                                                             const float* __restrict__ v_prev, int N, Segs n_cache,
                                                             float2* __restrict__ va, float4* __restrict__ partial,
                                                             int chunks) {
  __shared__ float4 red[kStatThreads / 64];
  const int b = blockIdx.y, chunk = blockIdx.x;
  if (n_cache.off[b] == 0) return;
  const int tid = threadIdx.x;
  const size_t base = (size_t)b * N;
  float4 c0[kStatPer], c1[kStatPer], p0[kStatPer], p1[kStatPer];
#pragma unroll
  for (int j = 0; j < kStatPer; ++j) {
    const int i = min(chunk * kChunk + j * kStatThreads + tid, N - 1);   // clamped: loads stay in bounds
    const float4* pc = reinterpret_cast<const float4*>(v_cache + (base + i) * 8);
    const float4* pp = reinterpret_cast<const float4*>(v_prev + (base + i) * 8);
    c0[j] = pc[0];
    c1[j] = pc[1];
    p0[j] = pp[0];
    p1[j] = pp[1];
  }
  float loV = INFINITY, hiV = -INFINITY, loA = INFINITY, hiA = -INFINITY;
#pragma unroll
  for (int j = 0; j < kStatPer; ++j) {
    const int i = chunk * kChunk + j * kStatThreads + tid;
    if (i < N) {
      const float V = sqrt_rn(sumsq8(c0[j], c1[j]));
      const float A = sqrt_rn(sumsq8(sub4(c0[j], p0[j]), sub4(c1[j], p1[j])));
      va[base + i] = make_float2(V, A);
      loV = fminf(loV, V);
      hiV = fmaxf(hiV, V);
      loA = fminf(loA, A);
      hiA = fmaxf(hiA, A);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    loV = fminf(loV, __shfl_xor(loV, o));
    hiV = fmaxf(hiV, __shfl_xor(hiV, o));
    loA = fminf(loA, __shfl_xor(loA, o));
    hiA = fmaxf(hiA, __shfl_xor(hiA, o));
  }
  if ((tid & 63) == 0) red[tid >> 6] = make_float4(loV, hiV, loA, hiA);
  __syncthreads();
  if (tid == 0) {
    float4 m = red[0];
#pragma unroll
    for (int w = 1; w < kStatThreads / 64; ++w) {
      m.x = fminf(m.x, red[w].x);
      m.y = fmaxf(m.y, red[w].y);
      m.z = fminf(m.z, red[w].z);
      m.w = fmaxf(m.w, red[w].w);
    }
    partial[(size_t)b * chunks + chunk] = m;
  }
}

// FROM_SCORES: the keys come from caller-given scores (given [B][N]) instead
// of the magnitude pairs; everything after the keys is the same.
template <bool FROM_SCORES>
__global__ __launch_bounds__(kThreads) void k_select(const float2* __restrict__ va, const float4* __restrict__ partial,
                                                     int chunks, int N, float w_a, float w_v, Segs n_cache, Segs act,
                                                     int32_t* __restrict__ idx_active, int32_t* __restrict__ pos,
                                                     float* __restrict__ score, const float* __restrict__ given) {
  __shared__ uint32_t keys[kMaxTokens];
  __shared__ int hist[256];
  __shared__ int cnt_eq[kMaxTokens / 64], cnt_act[kMaxTokens / 64];   // per (round, wave)
  __shared__ int sel[2];
  __shared__ float4 ext;

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int c = n_cache.off[b];
  const int row0 = act.off[b];
  const size_t base = (size_t)b * N;
  const int lane = tid & 63, wave = tid >> 6;

  if (c == 0) {  // full step for this sample: identity selection, no scoring
    for (int i = tid; i < N; i += kThreads) {
      idx_active[row0 + i] = i;
      pos[base + i] = row0 + i;
    }
    return;
  }

  if constexpr (FROM_SCORES) {
    for (int i = tid; i < N; i += kThreads) keys[i] = order_key(given[base + i]);
  } else {
    // The sample's extremes from the partials (chunks <= 64: one wave).
    if (wave == 0) {
      float4 m = lane < chunks ? partial[(size_t)b * chunks + lane]
                               : make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        m.x = fminf(m.x, __shfl_xor(m.x, o));
        m.y = fmaxf(m.y, __shfl_xor(m.y, o));
        m.z = fminf(m.z, __shfl_xor(m.z, o));
        m.w = fmaxf(m.w, __shfl_xor(m.w, o));
      }
      if (lane == 0) ext = m;
    }
    __syncthreads();
    const float loV = ext.x, hiV = ext.y, loA = ext.z, hiA = ext.w;

    // Scores and order keys.
    for (int i = tid; i < N; i += kThreads) {
      const float2 p = va[base + i];
      const float cs = __fadd_rn(__fmul_rn(w_a, norm_term(p.y, loA, hiA)), __fmul_rn(w_v, norm_term(p.x, loV, hiV)));
      keys[i] = order_key(cs);
      if (score) score[base + i] = cs;
    }
  }
  __syncthreads();

  // Radix select of the key with 0-based rank c-1. The keys of one sample
  // mostly share their leading byte (scores lie in [0, 1]), so a wave first
  // merges the lanes that share the bin of its lowest pending lane, twice,
  // with one LDS atomic per merged bin (same-address atomics of one
  // instruction would serialise); the lanes left add their own key.
  const uint64_t below = (1ull << lane) - 1ull;   // lanes before this one
  uint32_t prefix = 0, mask = 0;
  int r = c;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kThreads) hist[i] = 0;
    __syncthreads();
    for (int i0 = 0; i0 < N; i0 += kThreads) {     // whole waves iterate together (ballots below)
      const int i = i0 + tid;
      const uint32_t k = i < N ? keys[i] : 0u;
      const bool in = i < N && (k & mask) == prefix;
      const int bin = (int)((k >> shift) & 255u);
      uint64_t todo = __ballot(in);
#pragma unroll
      for (int it = 0; it < 2; ++it) {
        if (!todo) break;
        const int leader = __ffsll((unsigned long long)todo) - 1;
        const int lb = __shfl(bin, leader);
        const uint64_t same = __ballot(in && bin == lb);
        if (lane == leader) atomicAdd(&hist[lb], __popcll(same));
        todo &= ~same;
      }
      if ((todo >> lane) & 1ull) atomicAdd(&hist[bin], 1);
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

  // Token-order scan. Token i = 1024 j + 64 w + lane is handled by lane
  // `lane` of wave w in round j, so (j, w, lane) runs in token order. A token
  // is cached when its key is below kstar, or equal and among the first r
  // equal keys. Per (round, wave) counts of equal keys, then of active
  // tokens, go through an exclusive scan in LDS; a lane's rank inside its
  // wave is the popcount of the ballot below it. Loads and stores of one
  // wave touch 64 consecutive tokens.
  const int rounds = (N + kThreads - 1) / kThreads;
  const int nw = kThreads / 64;
  for (int j = 0; j < rounds; ++j) {
    const int i = j * kThreads + tid;
    const uint64_t eq = __ballot(i < N && keys[i] == kstar);
    if (lane == 0) cnt_eq[j * nw + wave] = __popcll(eq);
  }
  __syncthreads();
  segment_exclusive_scan(cnt_eq, rounds * nw, lane, wave);
  __syncthreads();
  for (int j = 0; j < rounds; ++j) {
    const int i = j * kThreads + tid;
    const uint32_t k = i < N ? keys[i] : 0xFFFFFFFFu;
    const bool is_eq = i < N && k == kstar;
    const uint64_t eq = __ballot(is_eq);
    const bool cached = k < kstar || (is_eq && cnt_eq[j * nw + wave] + __popcll(eq & below) < r);
    const uint64_t act_mask = __ballot(i < N && !cached);
    if (lane == 0) cnt_act[j * nw + wave] = __popcll(act_mask);
  }
  __syncthreads();
  segment_exclusive_scan(cnt_act, rounds * nw, lane, wave);
  __syncthreads();
  for (int j = 0; j < rounds; ++j) {
    const int i = j * kThreads + tid;
    const uint32_t k = i < N ? keys[i] : 0xFFFFFFFFu;
    const bool is_eq = i < N && k == kstar;
    const uint64_t eq = __ballot(is_eq);
    const bool cached = k < kstar || (is_eq && cnt_eq[j * nw + wave] + __popcll(eq & below) < r);
    const bool active = i < N && !cached;
    const uint64_t act_mask = __ballot(active);
    if (i < N) {
      const int a = row0 + cnt_act[j * nw + wave] + __popcll(act_mask & below);
      pos[base + i] = active ? a : -1;
      if (active) idx_active[a] = i;
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

// Static selection scratch for callers that cannot allocate (the no-alloc
// operator entry). Each device holds its own copy; its device address is
// looked up once per device and kept, since host code must never pass the
// symbol itself to a kernel.
constexpr size_t kStaticScratchBytes = (size_t(4) << 20) + (size_t(16) << 10);
static __device__ __align__(256) char scratch[kStaticScratchBytes];

hipError_t select_static_scratch(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static std::vector<void*> by_device;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)by_device.size() <= dev) by_device.resize(dev + 1, nullptr);
  if (!by_device[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    by_device[dev] = p;
  }
  *ptr = by_device[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

size_t select_workspace_bytes(int B, int N) {
  const int chunks = (N + kChunk - 1) / kChunk;
  return (((size_t)B * N * sizeof(float2) + 255) & ~(size_t)255) + (size_t)B * chunks * sizeof(float4);
}

hipError_t launch_select(const float* v_cache, const float* v_prev, int B, int N, float w_a, float w_v,
                         const Segs& n_cache, const Segs& act, int32_t* idx_active, int32_t* pos,
                         float* score, void* workspace, hipStream_t s) {
  const int chunks = (N + kChunk - 1) / kChunk;
  float2* va = static_cast<float2*>(workspace);
  float4* partial = reinterpret_cast<float4*>(static_cast<char*>(workspace) +
                                              (((size_t)B * N * sizeof(float2) + 255) & ~(size_t)255));
  launch(k_score_stats, dim3(chunks, B), dim3(kStatThreads), 0, s, v_cache, v_prev, N, n_cache, va, partial, chunks);
  launch(k_select<false>, dim3(B), dim3(kThreads), 0, s, (const float2*)va, (const float4*)partial, chunks, N, w_a,
         w_v, n_cache, act, idx_active, pos, score, (const float*)nullptr);
  return hipGetLastError();
}

hipError_t launch_select_scores(const float* scores, int B, int N, const Segs& n_cache, const Segs& act,
                                int32_t* idx_active, int32_t* pos, hipStream_t s) {
  launch(k_select<true>, dim3(B), dim3(kThreads), 0, s, (const float2*)nullptr, (const float4*)nullptr, 0, N, 0.0f,
         0.0f, n_cache, act, idx_active, pos, (float*)nullptr, scores);
  return hipGetLastError();
}

}  // namespace f3c
