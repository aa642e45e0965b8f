// Variable-length multi-head softmax attention on the 32x32 matrix cores, used
// for self-attention over the active tokens of each sample (Sec. 4.2: self
// attention runs on the active subset only) and for cross-attention from the
// active tokens to the image-condition tokens.
//
// Online softmax over key/value tiles of 64 staged in LDS (V is stored
// transposed). Each wavefront owns 32 queries and computes S^T = K Q^T, so a
// lane holds one query's scores for 16 of every 32 keys: the running max and
// sum are per-lane values combined with a single cross-half exchange
// (lane l with l ^ 32). The same accumulator layout feeds O^T = V^T P^T as the
// B operand without any data movement; the K-slot order of P (keys
// 8*(e/4) + 4*(l/32) + e%4) is matched when the V^T fragment is read.
#include "common.h"
#include "kernels.h"

namespace f3c {

namespace {

constexpr int kBQ = 128;    // queries per workgroup (4 waves x 32)
constexpr int kBKV = 64;    // keys per LDS tile

struct AttnArgs {
  Segs qs, ks;
  int tile_off[kMaxBatch + 1];   // prefix of query tiles per sample
  const char* q;
  const char* k;
  const char* v;
  char* o;
  int ldq, ldk, ldv, ldo;        // elements
  float scale_log2;              // log2(e) / sqrt(hd)
};

template <typename T, int HD, int SITE>
__global__ __launch_bounds__(256) void k_attn(AttnArgs p) {
  constexpr int ES = sizeof(T);
  constexpr int E = Mfma<T>::E;
  constexpr int KRS = HD * ES + 16;          // K tile row stride (bytes)
  constexpr int VRS = kBKV * ES + 8;         // V^T tile row stride (bytes)
  constexpr int NKS = HD * ES / 32;          // 32-byte K slices over the head dim
  constexpr int PER16 = 16 / ES;
  constexpr int MMA_PER_READ = PER16 / E;
  constexpr int HT = HD / 32;                // 32-row output tiles over the head dim
  constexpr int CH = kBKV * HD * ES / 16;    // 16-byte chunks per K (or V) tile
  __shared__ __attribute__((aligned(16))) char Ks[kBKV * KRS];
  __shared__ __attribute__((aligned(16))) char Vt[HD * VRS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, r32 = lane & 31;
  const int head = blockIdx.y;
  const int b = find_segment(p.tile_off, p.qs.B, blockIdx.x);
  const int qt = blockIdx.x - p.tile_off[b];
  const int q_begin = p.qs.off[b], nq = p.qs.off[b + 1] - q_begin;
  const int k_begin = p.ks.off[b], nk = p.ks.off[b + 1] - k_begin;
  const int qi = qt * kBQ + wave * 32 + r32;          // query of this lane (within the sample)
  const bool q_ok = qi < nq;

  // Q^T as the B operand: lane reads 16 bytes of its query row per 32-byte slice.
  u32x4 qf[NKS];
  {
    const char* qrow = p.q + ((size_t)(q_begin + (q_ok ? qi : 0)) * p.ldq + head * HD) * ES;
#pragma unroll
    for (int s = 0; s < NKS; ++s)
      qf[s] = q_ok ? *reinterpret_cast<const u32x4*>(qrow + s * 32 + g * 16) : u32x4{0, 0, 0, 0};
  }

  f32x16 oacc[HT];
#pragma unroll
  for (int t = 0; t < HT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[t][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  const float c = p.scale_log2;

  for (int kv0 = 0; kv0 < nk; kv0 += kBKV) {
    // Stage K (row-major) and V (transposed) for keys kv0 .. kv0+63.
#pragma unroll
    for (int q = 0; q < CH / 256; ++q) {
      const int ch = tid + 256 * q;
      const int row = ch / (HD * ES / 16), col = ch % (HD * ES / 16);
      const bool ok = kv0 + row < nk;
      const size_t key = (size_t)(k_begin + kv0 + row);
      u32x4 kk = ok ? *reinterpret_cast<const u32x4*>(p.k + (key * p.ldk + head * HD) * ES + col * 16)
                    : u32x4{0, 0, 0, 0};
      u32x4 vv = ok ? *reinterpret_cast<const u32x4*>(p.v + (key * p.ldv + head * HD) * ES + col * 16)
                    : u32x4{0, 0, 0, 0};
      *reinterpret_cast<u32x4*>(Ks + row * KRS + col * 16) = kk;
      const T* ve = reinterpret_cast<const T*>(&vv);
#pragma unroll
      for (int e = 0; e < PER16; ++e) *reinterpret_cast<T*>(Vt + (col * PER16 + e) * VRS + row * ES) = ve[e];
    }
    __syncthreads();

    // S^T tiles: rows = keys kv0 + 32*kt + ..., cols = this wave's 32 queries.
    f32x16 sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kt][e] = 0.0f;
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const u32x4 kf = *reinterpret_cast<const u32x4*>(Ks + (kt * 32 + r32) * KRS + s * 32 + g * 16);
#pragma unroll
        for (int u = 0; u < MMA_PER_READ; ++u) {
          typename Mfma<T>::frag a, bq;
          if constexpr (ES == 2) {
            a = __builtin_bit_cast(bf16x8, kf);
            bq = __builtin_bit_cast(bf16x8, qf[s]);
          } else {
            a = __builtin_bit_cast(f32x4, kf)[u];
            bq = __builtin_bit_cast(f32x4, qf[s])[u];
          }
          sacc[kt] = Mfma<T>::mma(a, bq, sacc[kt]);
        }
      }
    }

    // Online softmax (base 2). Key of element e: kv0 + 32*kt + 8*(e/4) + 4*g + e%4.
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = kv0 + kt * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
        if (key >= nk) sacc[kt][e] = -INFINITY;
        mx = fmaxf(mx, sacc[kt][e]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
    const float mc = m_new * c;
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int t = 0; t < HT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[t][e] *= alpha;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float pe = __builtin_amdgcn_exp2f(fmaf(sacc[kt][e], c, -mc));
        sacc[kt][e] = pe;
        l_run += pe;
      }

    // O^T += V^T P^T over the 64 keys.
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int u = 0; u < 16 / E; ++u) {
        typename Mfma<T>::frag pf;
        if constexpr (ES == 2) {
#pragma unroll
          for (int e = 0; e < 8; ++e) pf[e] = (bf16)sacc[kt][8 * u + e];
        } else {
          pf = sacc[kt][u];
        }
#pragma unroll
        for (int t = 0; t < HT; ++t) {
          const char* vrow = Vt + (t * 32 + r32) * VRS;
          typename Mfma<T>::frag vf;
          if constexpr (ES == 2) {
            const int key0 = kt * 32 + 16 * u + 4 * g;
            const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + key0 * ES);
            const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + (key0 + 8) * ES);
            vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
          } else {
            const int key = kt * 32 + 8 * (u >> 2) + 4 * g + (u & 3);
            vf = *reinterpret_cast<const float*>(vrow + key * ES);
          }
          oacc[t] = Mfma<T>::mma(vf, pf, oacc[t]);
        }
      }
    __syncthreads();
  }

  if (!q_ok) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.0f / l_tot;
  T* orow = reinterpret_cast<T*>(p.o + ((size_t)(q_begin + qi) * p.ldo + head * HD) * ES);
#pragma unroll
  for (int t = 0; t < HT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) orow[t * 32 + 8 * (e >> 2) + 4 * g + (e & 3)] = from_f32<T>(oacc[t][e] * inv);
}

template <int SITE>
hipError_t launch_a(int dt, int hd, dim3 grid, const AttnArgs& a, hipStream_t s) {
  if (dt == DT_BF16 && hd == 64) hipLaunchKernelGGL((k_attn<bf16, 64, SITE>), grid, dim3(256), 0, s, a);
  else if (dt == DT_BF16 && hd == 32) hipLaunchKernelGGL((k_attn<bf16, 32, SITE>), grid, dim3(256), 0, s, a);
  else if (dt == DT_F32 && hd == 64) hipLaunchKernelGGL((k_attn<float, 64, SITE>), grid, dim3(256), 0, s, a);
  else if (dt == DT_F32 && hd == 32) hipLaunchKernelGGL((k_attn<float, 32, SITE>), grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int site, int dt, int heads, int hd, const Segs& qs, const Segs& ks, const void* q,
                            int ldq, const void* k, int ldk, const void* v, int ldv, void* o, int ldo, hipStream_t s) {
  AttnArgs a;
  a.qs = qs;
  a.ks = ks;
  a.tile_off[0] = 0;
  for (int b = 0; b < qs.B; ++b) a.tile_off[b + 1] = a.tile_off[b] + (qs.off[b + 1] - qs.off[b] + kBQ - 1) / kBQ;
  const int tiles = a.tile_off[qs.B];
  if (tiles == 0) return hipSuccess;
  a.q = (const char*)q;
  a.k = (const char*)k;
  a.v = (const char*)v;
  a.o = (char*)o;
  a.ldq = ldq;
  a.ldk = ldk;
  a.ldv = ldv;
  a.ldo = ldo;
  a.scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  dim3 grid(tiles, heads);
  if (site == SITE_SELF) return launch_a<SITE_SELF>(dt, hd, grid, a, s);
  if (site == SITE_CROSS) return launch_a<SITE_CROSS>(dt, hd, grid, a, s);
  return launch_a<SITE_OP>(dt, hd, grid, a, s);
}

}  // namespace f3c
