// Row-wise and element-wise kernels of the cached step: active-token gather +
// input embedding, LayerNorm with adaLN modulation, final LayerNorm + output
// projection, merge + Euler + cache rotation, the timestep/modulation GEMVs
// and dtype conversion. All are HBM/latency bound; one 64-wide wavefront owns a
// row and lanes stride across the row so every load instruction is coalesced.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace f3c {

namespace {

constexpr float kLnEps = 1e-6f;

// ---------------------------------------------------------------- gather + embed
// h[r][n] = sum_c x[b][i][c] * W_in[n][c] + b_in[n] + P[i][n]   (Sec. 4.2 index-based
// selection: x_active = x[:, I_active, :], positions travel with the token).
template <typename T, int NPL>
__global__ __launch_bounds__(256) void k_embed(const float* __restrict__ x, int N, const int32_t* __restrict__ idx,
                                               Segs act, const T* __restrict__ w_in,
                                               const float* __restrict__ b_in, const T* __restrict__ ptab,
                                               float* __restrict__ h, int64_t dup) {
  constexpr int D = NPL * 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int total = act.off[act.B];
  if (row >= total) return;
  const int b = find_segment(act.off, act.B, row);
  const int i = idx ? idx[row] : row - act.off[b];
  const float* xr = x + ((size_t)b * N + i) * 8;
  float xv[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) xv[c] = xr[c];
  const T* pr = ptab + (size_t)i * D;
  float* hr = h + (size_t)row * D;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int n = lane + 64 * j;
    const T* w = w_in + (size_t)n * 8;
    float acc = 0.0f;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc += xv[c] * to_f32(w[c]);
    const float e = acc + b_in[n] + to_f32(pr[n]);
    hr[n] = e;
    if (dup) hr[dup * D + n] = e;           // the unconditional pass's copy of the row
  }
}

// The same for bf16 models with d a multiple of 256, streaming rows. A row is
// split over WPR waves (WPR divides G = d / 256, the column groups of 256);
// lane l of a wave owns columns 256 g + 4 l .. +3 of its GPW = G / WPR groups
// and keeps their input weights (packed bf16) and biases in registers, so a
// row costs only its 32-byte x row (one address per wave), its bf16 position
// row (8-byte loads) and its f32 output row (16-byte stores). Wave w handles
// part w % WPR of rows w / WPR + k * walkers, U rows per round; the token
// indices of the next round are loaded while the current round's rows are
// fetched, so each round waits for one memory round trip. Same operation
// order as k_embed. Four rows per round measured best on MI355X at d = 1024
// (9830 of 32768 tokens: 12.7 against 14.2 us with eight; all 32768: 29.3
// against 31.8 us; four samples of 9830: 37.9 against 42.4 us).
template <int G, int WPR, int U = 4>
__global__ __launch_bounds__(256) void k_embed_rows(const float* __restrict__ x, int N, const int32_t* __restrict__ idx,
                                                    Segs act, const bf16* __restrict__ w_in,
                                                    const float* __restrict__ b_in, const bf16* __restrict__ ptab,
                                                    float* __restrict__ h, int64_t dup) {
  constexpr int D = G * 256;
  constexpr int GPW = G / WPR;
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int part = gw % WPR;
  const int walkers = gridDim.x * 4 / WPR;       // waves per part
  const int total = act.off[act.B];
  const int first = gw / WPR;
  // token of row r (idx may be null: identity within the segment), and its sample
  auto token = [&](int r, int& b) {
    b = find_segment(act.off, act.B, r);
    return idx ? idx[r] : r - act.off[b];
  };
  int nb[U], ni[U];
#pragma unroll
  for (int u = 0; u < U; ++u) ni[u] = token(min(first + u * walkers, total - 1), nb[u]);
  bf16x8 w[GPW][4];
  float4 bias[GPW];
#pragma unroll
  for (int g = 0; g < GPW; ++g) {
    const int n0 = 256 * (part * GPW + g) + 4 * lane;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[g][e] = *reinterpret_cast<const bf16x8*>(w_in + (size_t)(n0 + e) * 8);
    bias[g] = *reinterpret_cast<const float4*>(b_in + n0);
  }
  for (int r0 = first; r0 < total; r0 += U * walkers) {
    float xv[U][8];
    bf16x4 pv[U][GPW];
#pragma unroll
    for (int u = 0; u < U; ++u) {     // rows past the end repeat the last one (loads only)
      const float4* xr = reinterpret_cast<const float4*>(x + ((size_t)nb[u] * N + ni[u]) * 8);
      const float4 x0 = xr[0], x1 = xr[1];
      xv[u][0] = x0.x; xv[u][1] = x0.y; xv[u][2] = x0.z; xv[u][3] = x0.w;
      xv[u][4] = x1.x; xv[u][5] = x1.y; xv[u][6] = x1.z; xv[u][7] = x1.w;
#pragma unroll
      for (int g = 0; g < GPW; ++g)
        pv[u][g] = *reinterpret_cast<const bf16x4*>(ptab + (size_t)ni[u] * D + 256 * (part * GPW + g) + 4 * lane);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) ni[u] = token(min(r0 + (U + u) * walkers, total - 1), nb[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = r0 + u * walkers;
      if (row >= total) break;
      float* hr = h + (size_t)row * D;
#pragma unroll
      for (int g = 0; g < GPW; ++g) {
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float acc = 0.0f;
#pragma unroll
          for (int c = 0; c < 8; ++c) acc += xv[u][c] * static_cast<float>(w[g][e][c]);
          o[e] = acc + (&bias[g].x)[e] + static_cast<float>(pv[u][g][e]);
        }
        const float4 v = make_float4(o[0], o[1], o[2], o[3]);
        const int col = 256 * (part * GPW + g) + 4 * lane;
        *reinterpret_cast<float4*>(hr + col) = v;
        if (dup) *reinterpret_cast<float4*>(hr + dup * D + col) = v;
      }
    }
  }
}

// ------------------------------------------------------------- LayerNorm (+mod)
template <int NPL>
__device__ __forceinline__ void row_stats(const float (&v)[NPL], float& mean, float& rstd) {
  constexpr int D = NPL * 64;
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) s += v[j];
  mean = wave_sum(s) * (1.0f / D);
  float q = 0.0f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const float c = v[j] - mean;
    q += c * c;
  }
  rstd = rsqrtf(wave_sum(q) * (1.0f / D) + kLnEps);
}

template <typename T, int NPL>
__global__ __launch_bounds__(256) void k_ln_mod(const float* __restrict__ h, int rows,
                                                const float* __restrict__ shift, const float* __restrict__ scale,
                                                T* __restrict__ out) {
  constexpr int D = NPL * 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* hr = h + (size_t)row * D;
  T* o = out + (size_t)row * D;
  if constexpr (NPL % 4 == 0) {
    // 16-byte loads: lane owns elements 4*(lane + 64 j) .. +3.
    constexpr int NV = NPL / 4;
    float4 v[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) v[j] = reinterpret_cast<const float4*>(hr)[lane + 64 * j];
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j) sum += (v[j].x + v[j].y) + (v[j].z + v[j].w);
    const float mean = wave_sum(sum) * (1.0f / D);
    float sq = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const float a = v[j].x - mean, b = v[j].y - mean, c = v[j].z - mean, d = v[j].w - mean;
      sq += (a * a + b * b) + (c * c + d * d);
    }
    const float rstd = rsqrtf(wave_sum(sq) * (1.0f / D) + kLnEps);
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int n = 4 * (lane + 64 * j);
      float u[4] = {(v[j].x - mean) * rstd, (v[j].y - mean) * rstd, (v[j].z - mean) * rstd, (v[j].w - mean) * rstd};
      if (scale) {
        const float4 sc = *reinterpret_cast<const float4*>(scale + n);
        const float4 sh = *reinterpret_cast<const float4*>(shift + n);
        u[0] = u[0] * (1.0f + sc.x) + sh.x;
        u[1] = u[1] * (1.0f + sc.y) + sh.y;
        u[2] = u[2] * (1.0f + sc.z) + sh.z;
        u[3] = u[3] * (1.0f + sc.w) + sh.w;
      }
      if constexpr (sizeof(T) == 2) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (bf16)u[e];
        *reinterpret_cast<bf16x4*>(o + n) = w;
      } else {
        *reinterpret_cast<float4*>(o + n) = make_float4(u[0], u[1], u[2], u[3]);
      }
    }
  } else {
    float v[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) v[j] = hr[lane + 64 * j];
    float mean, rstd;
    row_stats<NPL>(v, mean, rstd);
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int n = lane + 64 * j;
      float u = (v[j] - mean) * rstd;
      if (scale) u = u * (1.0f + scale[n]) + shift[n];
      o[n] = from_f32<T>(u);
    }
  }
}

// ------------------------------------------------------ final norm + projection
template <typename T, int NPL>
__global__ __launch_bounds__(256) void k_final(const float* __restrict__ h, int rows, const T* __restrict__ w_out,
                                               const float* __restrict__ b_out, float* __restrict__ v_act) {
  constexpr int D = NPL * 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* hr = h + (size_t)row * D;
  float v[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) v[j] = hr[lane + 64 * j];
  float mean, rstd;
  row_stats<NPL>(v, mean, rstd);
  float acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int n = lane + 64 * j;
    const float u = (v[j] - mean) * rstd;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] += u * to_f32(w_out[(size_t)c * D + n]);
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = wave_sum(acc[c]);
  if (lane < 8) {
    float r = acc[0];
#pragma unroll
    for (int c = 1; c < 8; ++c) r = (lane == c) ? acc[c] : r;
    v_act[(size_t)row * 8 + lane] = r + b_out[lane];
  }
}

// ------------------------------------------------------ merge + Euler + rotate
// Algorithm 1 state update: v = v_cache; v[I_active] = v_active; S <- S - (t - t') v;
// the new v is written to the other half of the cache ping-pong pair. On a
// guided step (v_unc set) the fresh velocity of an active row is
// ga * v_cond - gw * v_uncond, ga = fp32(1 + w), gw = fp32(w), each product
// and the difference rounded (classifier-free guidance).
__device__ __forceinline__ float4 guide4(float4 c, float4 u, float ga, float gw) {
  return make_float4(__fsub_rn(__fmul_rn(ga, c.x), __fmul_rn(gw, u.x)), __fsub_rn(__fmul_rn(ga, c.y), __fmul_rn(gw, u.y)),
                     __fsub_rn(__fmul_rn(ga, c.z), __fmul_rn(gw, u.z)), __fsub_rn(__fmul_rn(ga, c.w), __fmul_rn(gw, u.w)));
}

__global__ __launch_bounds__(256) void k_euler(float* __restrict__ x, const float* __restrict__ v_cache,
                                               const float* __restrict__ v_act, const float* __restrict__ v_unc,
                                               float ga, float gw, const int32_t* __restrict__ pos,
                                               Segs act, int B, int N, float dt, float* __restrict__ v_new) {
#pragma clang fp contract(off)
  const int64_t tok = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (tok >= (int64_t)B * N) return;
  const int b = (int)(tok / N);
  const int i = (int)(tok - (int64_t)b * N);
  const int p = pos ? pos[tok] : act.off[b] + i;
  const float4* src = reinterpret_cast<const float4*>(p >= 0 ? v_act + (size_t)p * 8 : v_cache + tok * 8);
  float4 v0 = src[0], v1 = src[1];
  if (v_unc && p >= 0) {
    const float4* un = reinterpret_cast<const float4*>(v_unc + (size_t)p * 8);
    v0 = guide4(v0, un[0], ga, gw);
    v1 = guide4(v1, un[1], ga, gw);
  }
  float4* xr = reinterpret_cast<float4*>(x + tok * 8);
  float4 x0 = xr[0], x1 = xr[1];
  x0.x = __fsub_rn(x0.x, __fmul_rn(dt, v0.x));
  x0.y = __fsub_rn(x0.y, __fmul_rn(dt, v0.y));
  x0.z = __fsub_rn(x0.z, __fmul_rn(dt, v0.z));
  x0.w = __fsub_rn(x0.w, __fmul_rn(dt, v0.w));
  x1.x = __fsub_rn(x1.x, __fmul_rn(dt, v1.x));
  x1.y = __fsub_rn(x1.y, __fmul_rn(dt, v1.y));
  x1.z = __fsub_rn(x1.z, __fmul_rn(dt, v1.z));
  x1.w = __fsub_rn(x1.w, __fmul_rn(dt, v1.w));
  xr[0] = x0;
  xr[1] = x1;
  float4* vn = reinterpret_cast<float4*>(v_new + tok * 8);
  vn[0] = v0;
  vn[1] = v1;
}

// ----------------------------------------------------------------------- GEMV
// y[r] = W[r] . f(x) + b[r] (optionally SiLU(y)). The input vector is staged in
// LDS once per workgroup (optionally through SiLU, or generated as the
// sinusoidal timestep features [cos(1000 t f_j), sin(1000 t f_j)],
// f_j = 10000^(-j/half), evaluated in fp64); each wavefront then streams one
// weight row with 16-byte loads. One row per wave: the 1024-row timestep MLP
// then spans 256 workgroups instead of a few waves walking rows one after the
// other at HBM latency each.
constexpr int kGemvRowsPerWave = 1;
constexpr int kGemvChunk = 8;               // times per pass of the batched modulation

template <typename T>
__global__ __launch_bounds__(256) void k_gemv(const T* __restrict__ W, const float* __restrict__ bias,
                                              const float* __restrict__ x, double t, int in_mode, int out_silu,
                                              int rows, int K, float* __restrict__ y) {
  extern __shared__ float xs[];
  for (int k = threadIdx.x; k < K; k += 256) {
    float v;
    if (in_mode == GEMV_IN_TIMESTEP) {
      const int half = K / 2;
      const int j = k < half ? k : k - half;
      const double arg = 1000.0 * t * pow(10000.0, -(double)j / half);
      v = (float)(k < half ? cos(arg) : sin(arg));
    } else {
      v = x[k];
      if (in_mode == GEMV_IN_SILU) v = silu(v);
    }
    xs[k] = v;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kGemvRowsPerWave;
  constexpr int V = 16 / sizeof(T);
  for (int rr = 0; rr < kGemvRowsPerWave; ++rr) {
    const int row = row0 + rr;
    if (row >= rows) return;
    const T* wr = W + (size_t)row * K;
    float acc = 0.0f;
    for (int k0 = lane * V; k0 < K; k0 += 64 * V) {
      if constexpr (sizeof(T) == 2) {
        const bf16x8 w = *reinterpret_cast<const bf16x8*>(wr + k0);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc += (float)w[e] * xs[k0 + e];
      } else {
        const float4 w = *reinterpret_cast<const float4*>(wr + k0);
        acc += w.x * xs[k0] + w.y * xs[k0 + 1] + w.z * xs[k0 + 2] + w.w * xs[k0 + 3];
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) {
      float r = acc + bias[row];
      y[row] = out_silu ? silu(r) : r;
    }
  }
}

// y[r] = sum_k Wt[k][r] SiLU(x[k]) + b[r] for a weight stored input-major
// (Wt [K][R]). Lane owns 16/sizeof(T) consecutive outputs and streams 16-byte
// rows of Wt, so no cross-lane reduction is needed; the 4 waves of a
// workgroup split K and combine their partial sums through LDS.
template <typename T>
__global__ __launch_bounds__(256) void k_gemv_t(const T* __restrict__ Wt, const float* __restrict__ bias,
                                                const float* __restrict__ x, int R, int K, float* __restrict__ y) {
  constexpr int V = 16 / sizeof(T);
  __shared__ float part[3][64 * V];
  __shared__ float xs[4096];
  for (int k = threadIdx.x; k < K; k += 256) xs[k] = silu(x[k]);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 64 * V + lane * V;
  const int kq = K / 4, k0 = wave * kq;
  float acc[V];
#pragma unroll
  for (int e = 0; e < V; ++e) acc[e] = 0.0f;
  if (r0 < R) {
    const T* w = Wt + (size_t)k0 * R + r0;
#pragma unroll 8
    for (int k = 0; k < kq; ++k) {
      const float xv = xs[k0 + k];
      if constexpr (sizeof(T) == 2) {
        const bf16x8 wv = *reinterpret_cast<const bf16x8*>(w + (size_t)k * R);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += (float)wv[e] * xv;
      } else {
        const float4 wv = *reinterpret_cast<const float4*>(w + (size_t)k * R);
        acc[0] += wv.x * xv;
        acc[1] += wv.y * xv;
        acc[2] += wv.z * xv;
        acc[3] += wv.w * xv;
      }
    }
  }
  if (wave > 0) {
#pragma unroll
    for (int e = 0; e < V; ++e) part[wave - 1][lane * V + e] = acc[e];
  }
  __syncthreads();
  if (wave == 0 && r0 < R) {
#pragma unroll
    for (int e = 0; e < V; ++e)
      y[r0 + e] = ((acc[e] + part[0][lane * V + e]) + (part[1][lane * V + e] + part[2][lane * V + e])) + bias[r0 + e];
  }
}

// The all-block modulation for up to kGemvChunk times in one pass over the
// input-major weight: each 16-byte weight load serves every time of the chunk.
// Per output the operations and their order are those of k_gemv_t (four
// sequential K quarters, combined as ((q0 + q1) + (q2 + q3)) + bias), so each
// time's result equals k_gemv_t's bit for bit. Rows of xs past nt are zero and
// their results are not stored.
template <typename T>
__global__ __launch_bounds__(256) void k_gemv_tn(const T* __restrict__ Wt, const float* __restrict__ bias,
                                                 const float* __restrict__ x, int ldx, int nt, int R, int K,
                                                 float* __restrict__ y, int ldy) {
  constexpr int V = 16 / sizeof(T), NT = kGemvChunk;
  __shared__ float part[3][64 * V];
  extern __shared__ float xs[];                     // [NT][K]
  for (int j = threadIdx.x; j < NT * K; j += 256) {
    const int i = j / K, k = j - i * K;
    xs[j] = i < nt ? silu(x[(size_t)i * ldx + k]) : 0.0f;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 64 * V + lane * V;
  const int kq = K / 4, k0 = wave * kq;
  float acc[NT][V];
#pragma unroll
  for (int i = 0; i < NT; ++i)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[i][e] = 0.0f;
  if (r0 < R) {
    // Sixteen weight loads in flight per wave, issued before any of them is
    // used (one wave per SIMD at this grid; left to itself the compiler waits
    // on each load right after issuing it). The order of the sums is unchanged.
    constexpr int U = 16;                           // K/4 is a multiple of 32
    const T* w = Wt + (size_t)k0 * R + r0;
    for (int kb = 0; kb < kq; kb += U) {
      u32x4 raw[U];
#pragma unroll
      for (int u = 0; u < U; ++u) raw[u] = *reinterpret_cast<const u32x4*>(w + (size_t)(kb + u) * R);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float wf[V];
        if constexpr (sizeof(T) == 2) {
          const bf16x8 wv = __builtin_bit_cast(bf16x8, raw[u]);
#pragma unroll
          for (int e = 0; e < 8; ++e) wf[e] = (float)wv[e];
        } else {
          const float4 wv = __builtin_bit_cast(float4, raw[u]);
          wf[0] = wv.x;
          wf[1] = wv.y;
          wf[2] = wv.z;
          wf[3] = wv.w;
        }
#pragma unroll
        for (int i = 0; i < NT; ++i) {
          const float xv = xs[i * K + k0 + kb + u];
#pragma unroll
          for (int e = 0; e < V; ++e) acc[i][e] += wf[e] * xv;
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    if (i >= nt) break;                             // nt is uniform: every wave takes every barrier
    if (wave > 0) {
#pragma unroll
      for (int e = 0; e < V; ++e) part[wave - 1][lane * V + e] = acc[i][e];
    }
    __syncthreads();
    if (wave == 0 && r0 < R) {
#pragma unroll
      for (int e = 0; e < V; ++e)
        y[(size_t)i * ldy + r0 + e] =
            ((acc[i][e] + part[0][lane * V + e]) + (part[1][lane * V + e] + part[2][lane * V + e])) + bias[r0 + e];
    }
    __syncthreads();
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_convert(const float* __restrict__ src, T* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = from_f32<T>(src[i]);
}

#define F3C_NPL_LAUNCH(d, KERNEL, T, grid, s, ...)                                        \
  do {                                                                                     \
    switch ((d) / 64) {                                                                    \
      case 2: launch((KERNEL<T, 2>), grid, dim3(256), 0, s, __VA_ARGS__); break;   \
      case 4: launch((KERNEL<T, 4>), grid, dim3(256), 0, s, __VA_ARGS__); break;   \
      case 8: launch((KERNEL<T, 8>), grid, dim3(256), 0, s, __VA_ARGS__); break;   \
      case 16: launch((KERNEL<T, 16>), grid, dim3(256), 0, s, __VA_ARGS__); break; \
      case 32: launch((KERNEL<T, 32>), grid, dim3(256), 0, s, __VA_ARGS__); break; \
      default: return hipErrorInvalidValue;                                                \
    }                                                                                      \
    return hipGetLastError();                                                              \
  } while (0)

}  // namespace

hipError_t launch_embed(int dt, const float* x, int N, const int32_t* idx, const Segs& act, const void* w_in,
                        const float* b_in, const void* pos_table, int d, float* h, int64_t dup, hipStream_t s) {
  const int rows = act.off[act.B];
  if (rows == 0) return hipSuccess;
  dim3 grid((rows + 3) / 4);
  if (dt == DT_BF16 && d % 256 == 0 && d <= 2048) {
    // streaming rows, 4 per round; at most 768 workgroups (three per CU,
    // all resident at once)
    const int wpr = std::min(d / 256, 4);
    const int wgs = std::max(1, std::min((rows * wpr + 31) / 32, 768));
    const bf16* w = (const bf16*)w_in;
    const bf16* p = (const bf16*)pos_table;
    switch (d / 256) {
      case 1: launch(k_embed_rows<1, 1>, dim3(wgs), dim3(256), 0, s, x, N, idx, act, w, b_in, p, h, dup); break;
      case 2: launch(k_embed_rows<2, 2>, dim3(wgs), dim3(256), 0, s, x, N, idx, act, w, b_in, p, h, dup); break;
      case 4: launch(k_embed_rows<4, 4>, dim3(wgs), dim3(256), 0, s, x, N, idx, act, w, b_in, p, h, dup); break;
      case 8: launch(k_embed_rows<8, 4>, dim3(wgs), dim3(256), 0, s, x, N, idx, act, w, b_in, p, h, dup); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (dt == DT_BF16)
    F3C_NPL_LAUNCH(d, k_embed, bf16, grid, s, x, N, idx, act, (const bf16*)w_in, b_in, (const bf16*)pos_table, h,
                   dup);
  F3C_NPL_LAUNCH(d, k_embed, float, grid, s, x, N, idx, act, (const float*)w_in, b_in, (const float*)pos_table, h,
                 dup);
}

hipError_t launch_ln_mod(int dt, const float* h, int rows, int d, const float* shift, const float* scale, void* out,
                         hipStream_t s) {
  if (rows == 0) return hipSuccess;
  dim3 grid((rows + 3) / 4);
  if (dt == DT_BF16) F3C_NPL_LAUNCH(d, k_ln_mod, bf16, grid, s, h, rows, shift, scale, (bf16*)out);
  F3C_NPL_LAUNCH(d, k_ln_mod, float, grid, s, h, rows, shift, scale, (float*)out);
}

hipError_t launch_final(int dt, const float* h, int rows, int d, const void* w_out, const float* b_out,
                        float* v_act, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  dim3 grid((rows + 3) / 4);
  if (dt == DT_BF16) F3C_NPL_LAUNCH(d, k_final, bf16, grid, s, h, rows, (const bf16*)w_out, b_out, v_act);
  F3C_NPL_LAUNCH(d, k_final, float, grid, s, h, rows, (const float*)w_out, b_out, v_act);
}

// Zero fill with 16-byte stores: a kernel rather than a memset node, so that a
// caller may capture the state reset in a graph.
__global__ __launch_bounds__(256) void k_zero16(u32x4* __restrict__ p, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride) p[i] = u32x4{0, 0, 0, 0};
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  if (bytes % 16 || (uintptr_t)p % 16) return hipErrorInvalidValue;
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n16 + 255) / 256, 2048);
  launch(k_zero16, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<u32x4*>(p), n16);
  return hipGetLastError();
}

hipError_t launch_euler(float* x, const float* v_cache, const float* v_act, const float* v_unc, float ga, float gw,
                        const int32_t* pos, const Segs& act, int B, int N, float dt, float* v_new, hipStream_t s) {
  const int64_t n = (int64_t)B * N;
  if (n == 0) return hipSuccess;
  launch(k_euler, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, v_cache, v_act, v_unc, ga, gw, pos, act, B,
         N, dt, v_new);
  return hipGetLastError();
}

hipError_t launch_gemv(int dt, const void* W, const float* bias, const float* x, double t, int in_mode,
                       int out_silu, int rows, int K, float* y, hipStream_t s) {
  const int per_block = 4 * kGemvRowsPerWave;
  dim3 grid((rows + per_block - 1) / per_block);
  const size_t lds = (size_t)K * sizeof(float);
  if (dt == DT_BF16)
    launch(k_gemv<bf16>, grid, dim3(256), lds, s, (const bf16*)W, bias, x, t, in_mode, out_silu, rows,
                       K, y);
  else
    launch(k_gemv<float>, grid, dim3(256), lds, s, (const float*)W, bias, x, t, in_mode, out_silu,
                       rows, K, y);
  return hipGetLastError();
}

hipError_t launch_gemv_t(int dt, const void* Wt, const float* bias, const float* x, int R, int K, float* y,
                         hipStream_t s) {
  const int per_block = 64 * (dt == DT_BF16 ? 8 : 4);
  dim3 grid((R + per_block - 1) / per_block);
  if (dt == DT_BF16)
    launch(k_gemv_t<bf16>, grid, dim3(256), 0, s, (const bf16*)Wt, bias, x, R, K, y);
  else
    launch(k_gemv_t<float>, grid, dim3(256), 0, s, (const float*)Wt, bias, x, R, K, y);
  return hipGetLastError();
}

hipError_t launch_gemv_tn(int dt, const void* Wt, const float* bias, const float* x, int ldx, int nt, int R, int K,
                          float* y, int ldy, hipStream_t s) {
  if (nt < 1 || nt > kGemvChunk || K % 32) return hipErrorInvalidValue;
  const int per_block = 64 * (dt == DT_BF16 ? 8 : 4);
  dim3 grid((R + per_block - 1) / per_block);
  const size_t lds = (size_t)kGemvChunk * K * sizeof(float);
  if (dt == DT_BF16)
    launch(k_gemv_tn<bf16>, grid, dim3(256), lds, s, (const bf16*)Wt, bias, x, ldx, nt, R, K, y, ldy);
  else
    launch(k_gemv_tn<float>, grid, dim3(256), lds, s, (const float*)Wt, bias, x, ldx, nt, R, K, y, ldy);
  return hipGetLastError();
}

hipError_t launch_convert(int dt, const float* src, void* dst, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  dim3 grid((unsigned)(blocks < 65536 ? blocks : 65536));
  if (dt == DT_BF16)
    launch(k_convert<bf16>, grid, dim3(256), 0, s, src, (bf16*)dst, n);
  else
    launch(k_convert<float>, grid, dim3(256), 0, s, src, (float*)dst, n);
  return hipGetLastError();
}

}  // namespace f3c
