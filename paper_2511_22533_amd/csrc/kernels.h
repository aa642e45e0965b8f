// Internal launchers for the gfx950 kernels. Host code in f3c.cpp validates
// every shape before calling these; launchers only check launch errors.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace f3c {

constexpr int kMaxBatch = 64;          // samples per step (segment tables travel by value)
constexpr int kMaxTokens = 32768;      // tokens per sample (the selector keeps one sample's keys in LDS)

// Segment table passed by value: sample b owns rows [off[b], off[b+1]).
struct Segs {
  int B;
  int off[kMaxBatch + 1];
};

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };
enum Epilogue { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2 };

// Call sites of the dense kernels. Each site is its own template instance, so a
// kernel trace attributes time to the projection / attention it belongs to.
enum Site { SITE_OP = 0, SITE_QKV, SITE_O, SITE_Q, SITE_CO, SITE_FC1, SITE_FC2, SITE_COND, SITE_SELF, SITE_CROSS };

// Stability score + lowest-score selection: a streaming statistics pass over
// all tokens, then one workgroup per sample. v_cache, v_prev: f32 [B][N][8].
// n_cache: per-sample cached counts (by value). act: active-row offsets (by
// value). Writes idx_active[act.off[b] + r] (ascending token index of the r-th
// active token), pos[b*N + i] (packed row or -1) and, when score != nullptr,
// the float32 score of every token (only for c_b > 0). workspace (256-byte
// aligned, select_workspace_bytes(B, N) bytes) holds the per-token magnitude
// pairs and the per-workgroup extremes between the two kernels.
size_t select_workspace_bytes(int B, int N);
hipError_t launch_select(const float* v_cache, const float* v_prev, int B, int N, float w_a, float w_v,
                         const Segs& n_cache, const Segs& act, int32_t* idx_active, int32_t* pos,
                         float* score, void* workspace, hipStream_t s);
// The selection alone from caller-given float32 scores [B][N] (the same keys,
// radix select and token-order scan; no workspace).
hipError_t launch_select_scores(const float* scores, int B, int N, const Segs& n_cache, const Segs& act,
                                int32_t* idx_active, int32_t* pos, hipStream_t s);
// Device address and size of the selection's static scratch on the current
// device (looked up once per device, then cached).
hipError_t select_static_scratch(void** ptr, size_t* bytes);

// Teacher-forced selection: idx_out[r] = idx_in[r] (clamped into [0, N)) for
// the act.off[B] listed rows, pos[b][i] = r for listed tokens, -1 elsewhere.
hipError_t launch_force_active(const int32_t* idx_in, const Segs& act, int N, int32_t* idx_out, int32_t* pos,
                               hipStream_t s);

// h[r][:] = x[b][i][:] W_in^T + b_in + P[i][:], i = idx_active[r] (identity when idx == nullptr);
// with dup > 0 the row is also written to h[r + dup] (the unconditional pass of a guided step).
hipError_t launch_embed(int dt, const float* x, int N, const int32_t* idx, const Segs& act,
                        const void* w_in, const float* b_in, const void* pos_table, int d, float* h,
                        int64_t dup, hipStream_t s);

// out = LN(h) * (1 + scale) + shift, written as the model dtype; scale/shift may be null.
hipError_t launch_ln_mod(int dt, const float* h, int rows, int d, const float* shift, const float* scale,
                         void* out, hipStream_t s);

// v_act[r][c] = LN(h[r]) . W_out[c] + b_out[c], c < 8 (f32 output).
hipError_t launch_final(int dt, const float* h, int rows, int d, const void* w_out, const float* b_out,
                        float* v_act, hipStream_t s);

// Zero bytes (a multiple of 16) at p (16-byte aligned) with a kernel.
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

// Merge + Euler + rotate: v = (pos >= 0 ? v_act[pos] : v_cache); x -= dt * v; v_new = v.
// pos == nullptr means every token active at row act.off[b] + i. With v_unc (guided step), an
// active row's v is ga * v_act[p] - gw * v_unc[p], each operation rounded.
hipError_t launch_euler(float* x, const float* v_cache, const float* v_act, const float* v_unc, float ga,
                        float gw, const int32_t* pos, const Segs& act, int B, int N, float dt, float* v_new,
                        hipStream_t s);

// y[r] = W[r] . f(x) + b[r] (then SiLU when out_silu), f = identity / SiLU, or
// x := the K sinusoidal features of t. K must be a multiple of 16 / sizeof(element).
enum GemvIn { GEMV_IN_PLAIN = 0, GEMV_IN_SILU = 1, GEMV_IN_TIMESTEP = 2 };
hipError_t launch_gemv(int dt, const void* W, const float* bias, const float* x, double t, int in_mode,
                       int out_silu, int rows, int K, float* y, hipStream_t s);

// y[r] = sum_k Wt[k][r] SiLU(x[k]) + b[r] with the weight stored input-major
// (Wt [K][R]); R a multiple of 16 / sizeof(element), K a multiple of 4, K <= 4096.
hipError_t launch_gemv_t(int dt, const void* Wt, const float* bias, const float* x, int R, int K, float* y,
                         hipStream_t s);
// Up to 8 times at once: x [nt][ldx] (each time's t2 output), y [nt][ldy].
hipError_t launch_gemv_tn(int dt, const void* Wt, const float* bias, const float* x, int ldx, int nt, int R, int K,
                          float* y, int ldy, hipStream_t s);

// Element type conversion f32 -> model dtype.
hipError_t launch_convert(int dt, const float* src, void* dst, int64_t n, hipStream_t s);

// C = A W^T + bias with an epilogue. A: [M][lda], W: [N][ldw] (model dtype),
// bias f32 [N]. EPI_STORE / EPI_GELU write out[M][ldo] in the model dtype;
// EPI_RESID does resid[m][n] += (gate ? gate[n] : 1) * value in f32.
// Requires N % 128 == 0 and K % (128 / sizeof(element)) == 0. Each output is
// one workgroup's sum in a fixed order.
// EPI_STORE / EPI_GELU with oscale_cols > 0: output columns below oscale_cols
// are multiplied by oscale after the bias, before the store (the attention's
// pre-scaled queries).
hipError_t launch_gemm(int site, int dt, int epi, int M, int N, int K, const void* A, int lda, const void* W,
                       int ldw, const float* bias, const float* gate, void* out, int ldo, float* resid, int ldr,
                       hipStream_t s, float oscale = 1.0f, int oscale_cols = 0);

// Varlen multi-head softmax attention. Queries of sample b are rows
// [qs.off[b], qs.off[b+1]) of q; its keys/values are rows [ks.off[b], ks.off[b+1])
// of k and v. Head h uses columns [h*hd, (h+1)*hd). Output rows match queries.
// ws (f32, ws_bytes, 16-byte aligned) may be null; when present, launches
// with few query tiles split the key range and merge the splits through it.
// q_scaled: the queries were stored multiplied by attention_q_scale(hd)
// (the step's Q projections do so in their epilogue).
hipError_t launch_attention(int site, int dt, int heads, int hd, const Segs& qs, const Segs& ks, const void* q,
                            int ldq, const void* k, int ldk, const void* v, int ldv, void* o, int ldo, float* ws,
                            size_t ws_bytes, hipStream_t s, bool q_scaled = false);

// log2(e) / sqrt(hd): the softmax scale in base-2 units.
inline float attention_q_scale(int hd) { return 1.4426950408889634f / sqrtf((float)hd); }

// Occupancy bits from decoder logits (occupied when > 0) for B grids of
// n_voxels: bits [B][ceil(n_voxels / 32)] u32, voxel n in bit n % 32 of word n / 32.
hipError_t launch_pack_occupancy(const float* logits, int B, int64_t n_voxels, uint32_t* bits, hipStream_t s);

// counts[b] = popcount(a[b] ^ b[b]) over n_words words per grid (Eq. 1).
hipError_t launch_dynamic_voxels(const uint32_t* a, const uint32_t* b, int B, int64_t n_words, int64_t* counts,
                                 hipStream_t s);

}  // namespace f3c
