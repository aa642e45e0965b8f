// Dense projections of the transformer blocks on the 32x32 matrix cores:
// C = A W^T + bias, A = activations [M][K] (row-major, K contiguous),
// W = weights [N][K] (torch Linear layout, K contiguous), f32 accumulation.
// Epilogues fuse the bias with a dtype store (QKV / cross-attention Q / KV),
// GELU (tanh form, MLP fc1), or a gated residual update in f32
// (h += gate * (.), attention output projections and MLP fc2).
//
// Workgroup tile BM x BN, K staged 128 bytes at a time through padded LDS rows
// (144-byte stride: the 16-byte fragment reads of 8 consecutive lanes land on
// disjoint banks). 4 wavefronts in a 2 x 2 arrangement; each owns a
// (BM/2) x (BN/2) sub-tile of 32x32 MFMA accumulators. The next K tile is
// prefetched into registers while the current one is consumed from LDS.
// A lane reads 16 contiguous bytes of one row at K-group offset l/32; the same
// K mapping is used for A and W, so any assignment of K elements to the
// instruction's K slots gives the same dot products.
#include "common.h"
#include "kernels.h"

namespace f3c {

namespace {

constexpr int kBKB = 128;             // K bytes per LDS tile row
constexpr int kRS = kBKB + 16;        // padded LDS row stride (bytes)

struct GemmArgs {
  int M, N, K;
  const char* A;
  int lda;                            // elements
  const char* W;
  int ldw;
  const float* bias;
  const float* gate;
  void* out;
  int ldo;
  float* resid;
  int ldr;
};

template <typename T, int BM, int BN, int EPI, int SITE>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs p) {
  constexpr int TM = BM / 64, TN = BN / 64;                 // 32x32 tiles per wave
  constexpr int CA = BM * 8 / 256, CB = BN * 8 / 256;       // 16-byte chunks per thread
  constexpr int ES = sizeof(T);
  constexpr int PER16 = 16 / ES;                            // elements per 16 bytes
  constexpr int MMA_PER_READ = PER16 / Mfma<T>::E;          // instructions per fragment read
  __shared__ __attribute__((aligned(16))) char As[BM * kRS];
  __shared__ __attribute__((aligned(16))) char Bs[BN * kRS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 5, r32 = lane & 31;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const size_t lda_b = (size_t)p.lda * ES, ldw_b = (size_t)p.ldw * ES;

  u32x4 ra[CA], rb[CB];
  auto load_tile = [&](int kt) {
    const size_t kb = (size_t)kt * kBKB;
#pragma unroll
    for (int q = 0; q < CA; ++q) {
      const int c = tid + 256 * q, row = c >> 3, col = c & 7;
      const int m = m0 + row;
      if (m < p.M)
        ra[q] = *reinterpret_cast<const u32x4*>(p.A + (size_t)m * lda_b + kb + col * 16);
      else
        ra[q] = u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int q = 0; q < CB; ++q) {
      const int c = tid + 256 * q, row = c >> 3, col = c & 7;
      rb[q] = *reinterpret_cast<const u32x4*>(p.W + (size_t)(n0 + row) * ldw_b + kb + col * 16);
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int q = 0; q < CA; ++q) {
      const int c = tid + 256 * q, row = c >> 3, col = c & 7;
      *reinterpret_cast<u32x4*>(As + row * kRS + col * 16) = ra[q];
    }
#pragma unroll
    for (int q = 0; q < CB; ++q) {
      const int c = tid + 256 * q, row = c >> 3, col = c & 7;
      *reinterpret_cast<u32x4*>(Bs + row * kRS + col * 16) = rb[q];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int KT = (p.K * ES) / kBKB;
  load_tile(0);
  store_tile();
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) load_tile(kt + 1);
#pragma unroll
    for (int ks = 0; ks < kBKB / 32; ++ks) {
      u32x4 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const u32x4*>(As + (wm * (BM / 2) + i * 32 + r32) * kRS + ks * 32 + g * 16);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const u32x4*>(Bs + (wn * (BN / 2) + j * 32 + r32) * kRS + ks * 32 + g * 16);
#pragma unroll
      for (int u = 0; u < MMA_PER_READ; ++u)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            typename Mfma<T>::frag a, b;
            if constexpr (sizeof(T) == 2) {
              a = __builtin_bit_cast(bf16x8, fa[i]);
              b = __builtin_bit_cast(bf16x8, fb[j]);
            } else {
              a = __builtin_bit_cast(f32x4, fa[i])[u];
              b = __builtin_bit_cast(f32x4, fb[j])[u];
            }
            acc[i][j] = Mfma<T>::mma(a, b, acc[i][j]);
          }
    }
    __syncthreads();
    if (kt + 1 < KT) {
      store_tile();
      __syncthreads();
    }
  }

  // Epilogue: lane holds column r32 and rows 8*(e/4) + 4*g + e%4 of each tile.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * (BN / 2) + j * 32 + r32;
      const float bcol = p.bias[col];
      const float gcol = (EPI == EPI_RESID && p.gate) ? p.gate[col] : 1.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm * (BM / 2) + i * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
        if (row >= p.M) continue;
        const float v = acc[i][j][e] + bcol;
        if constexpr (EPI == EPI_RESID) {
          float* r = p.resid + (size_t)row * p.ldr + col;
          *r = *r + gcol * v;
        } else if constexpr (EPI == EPI_GELU) {
          reinterpret_cast<T*>(p.out)[(size_t)row * p.ldo + col] = from_f32<T>(gelu_tanh(v));
        } else {
          reinterpret_cast<T*>(p.out)[(size_t)row * p.ldo + col] = from_f32<T>(v);
        }
      }
    }
}

template <typename T, int EPI, int SITE>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
  constexpr int BM = 128, BN = 128;
  dim3 grid(a.N / BN, (a.M + BM - 1) / BM);
  hipLaunchKernelGGL((k_gemm<T, BM, BN, EPI, SITE>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_site(int site, int epi, const GemmArgs& a, hipStream_t s) {
  switch (site) {
    case SITE_QKV: return launch_t<T, EPI_STORE, SITE_QKV>(a, s);
    case SITE_Q: return launch_t<T, EPI_STORE, SITE_Q>(a, s);
    case SITE_COND: return launch_t<T, EPI_STORE, SITE_COND>(a, s);
    case SITE_O: return launch_t<T, EPI_RESID, SITE_O>(a, s);
    case SITE_CO: return launch_t<T, EPI_RESID, SITE_CO>(a, s);
    case SITE_FC2: return launch_t<T, EPI_RESID, SITE_FC2>(a, s);
    case SITE_FC1: return launch_t<T, EPI_GELU, SITE_FC1>(a, s);
    default: break;
  }
  switch (epi) {
    case EPI_STORE: return launch_t<T, EPI_STORE, SITE_OP>(a, s);
    case EPI_GELU: return launch_t<T, EPI_GELU, SITE_OP>(a, s);
    case EPI_RESID: return launch_t<T, EPI_RESID, SITE_OP>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(int site, int dt, int epi, int M, int N, int K, const void* A, int lda, const void* W,
                       int ldw, const float* bias, const float* gate, void* out, int ldo, float* resid, int ldr,
                       hipStream_t s) {
  if (M == 0) return hipSuccess;
  GemmArgs a{M, N, K, (const char*)A, lda, (const char*)W, ldw, bias, gate, out, ldo, resid, ldr};
  return dt == DT_BF16 ? launch_site<bf16>(site, epi, a, s) : launch_site<float>(site, epi, a, s);
}

}  // namespace f3c
