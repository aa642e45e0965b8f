// Dynamic voxels of the decoded occupancy grid (Eq. 1): the number of voxels
// whose binary occupancy differs between the grids decoded at two consecutive
// steps. The decoder's output (one logit per voxel, occupied when > 0) is
// packed 32 voxels per word, voxel n in bit n % 32 of word n / 32 (row-major
// flattening, zero-padded tail); the count is the popcount of the XOR of two
// packed grids. Both kernels are bound by HBM: 4 bytes read per voxel when
// packing, 2 x 1/8 byte per voxel when counting.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace f3c {

namespace {

constexpr int kGroups = 8;                     // dword path: 64-voxel groups per wave and pass
constexpr int kChunks = 4;                     // vector path: 256-voxel chunks per wave and pass

// Bits 0..7 of x moved to bits 0, 4, 8, ..., 28.
__device__ __forceinline__ uint32_t spread4(uint32_t x) {
  x = (x | (x << 12)) & 0x000F000Fu;
  x = (x | (x << 6)) & 0x03030303u;
  return (x | (x << 3)) & 0x11111111u;
}

// Vector path (rows 16-byte aligned, n_voxels % 4 == 0). A pass of a wave
// covers 4 chunks of 256 voxels; lane l loads voxels 4l..4l+3 of each chunk
// with one 16-byte load (all four loads issued together). Ballot k of a chunk
// holds component k of every lane: voxel 4l + k is bit l. Word j of the chunk
// (voxels 32j..32j+31, lanes 8j..8j+7) is therefore byte j of the four ballots
// interleaved bit by bit; lanes 0..31 build and store the pass's 32 words.
__global__ __launch_bounds__(256) void k_pack_occupancy_vec(const float* __restrict__ logits, int64_t n_voxels,
                                                            int64_t n_words, uint32_t* __restrict__ bits) {
  const int lane = threadIdx.x & 63;
  const f32x4* src = reinterpret_cast<const f32x4*>(logits + (size_t)blockIdx.y * n_voxels);
  uint32_t* dst = bits + (size_t)blockIdx.y * n_words;
  const int64_t n4 = n_voxels / 4;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int64_t n_pass = (n4 + 64 * kChunks - 1) / (64 * kChunks);
  const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); p < n_pass; p += waves) {
    const int64_t q0 = p * 64 * kChunks;       // first float4 of the pass
    f32x4 x[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int64_t q = q0 + c * 64 + lane;
      x[c] = q < n4 ? src[q] : zero;           // padding voxels are unoccupied
    }
    uint64_t m[4] = {0, 0, 0, 0};
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint64_t b = __builtin_amdgcn_ballot_w64(x[c][k] > 0.0f);   // NaN compares false
        if ((lane >> 3) == c) m[k] = b;
      }
    }
    const int sh = 8 * (lane & 7);
    uint32_t word = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) word |= spread4((uint32_t)(m[k] >> sh) & 0xFFu) << k;
    const int64_t w = q0 / 8 + lane;
    if (lane < 8 * kChunks && w < n_words) dst[w] = word;
  }
}

// Dword path (any alignment): passes of 8 x 64 consecutive voxels, eight
// coalesced 256-byte loads issued together, one ballot per 64 voxels (bit l =
// voxel 64g + l: words 2g and 2g + 1 of the pass); lanes 0..15 store.
__global__ __launch_bounds__(256) void k_pack_occupancy(const float* __restrict__ logits, int64_t n_voxels,
                                                        int64_t n_words, uint32_t* __restrict__ bits) {
  const int lane = threadIdx.x & 63;
  const float* src = logits + (size_t)blockIdx.y * n_voxels;
  uint32_t* dst = bits + (size_t)blockIdx.y * n_words;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int64_t n_pass = (n_voxels + 64 * kGroups - 1) / (64 * kGroups);
  for (int64_t p = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); p < n_pass; p += waves) {
    const int64_t v0 = p * 64 * kGroups;
    float x[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
      const int64_t v = v0 + g * 64 + lane;
      x[g] = v < n_voxels ? src[v] : 0.0f;     // padding voxels are unoccupied
    }
    uint32_t word = 0;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
      const uint64_t m = __builtin_amdgcn_ballot_w64(x[g] > 0.0f);   // NaN compares false: unoccupied
      if (lane == 2 * g) word = (uint32_t)m;
      if (lane == 2 * g + 1) word = (uint32_t)(m >> 32);
    }
    const int64_t w = v0 / 32 + lane;
    if (lane < 2 * kGroups && w < n_words) dst[w] = word;
  }
}

__global__ void k_zero_counts(int64_t* __restrict__ counts, int B) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < B) counts[i] = 0;
}

// popcount(a ^ b) over the words of sample blockIdx.y, split over gridDim.x
// workgroups. With one workgroup per sample it stores the count; otherwise
// each workgroup adds its partial sum to counts[b] (zeroed beforehand) with
// one 64-bit integer atomic, exact in any order.
template <bool VEC, bool ATOMIC>
__global__ __launch_bounds__(256) void k_dynamic_voxels(const uint32_t* __restrict__ a, const uint32_t* __restrict__ b,
                                                        int64_t n_words, int64_t* __restrict__ counts) {
  const size_t base = (size_t)blockIdx.y * n_words;
  const int64_t stride = (int64_t)gridDim.x * 256;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  uint64_t acc = 0;
  if constexpr (VEC) {                         // 16-byte aligned rows of a multiple of 4 words
    const u32x4* a4 = reinterpret_cast<const u32x4*>(a + base);
    const u32x4* b4 = reinterpret_cast<const u32x4*>(b + base);
    const int64_t n4 = n_words / 4;
    int64_t i = t;
    for (; i + 3 * stride < n4; i += 4 * stride) {
      u32x4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = a4[i + u * stride] ^ b4[i + u * stride];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc += __builtin_popcount(x[u][0]) + __builtin_popcount(x[u][1]) + __builtin_popcount(x[u][2]) +
               __builtin_popcount(x[u][3]);
    }
    for (; i < n4; i += stride) {
      const u32x4 x = a4[i] ^ b4[i];
      acc += __builtin_popcount(x[0]) + __builtin_popcount(x[1]) + __builtin_popcount(x[2]) +
             __builtin_popcount(x[3]);
    }
  } else {
    for (int64_t i = t; i < n_words; i += stride) acc += __builtin_popcount(a[base + i] ^ b[base + i]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  __shared__ uint64_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint64_t sum = part[0] + part[1] + part[2] + part[3];
    if constexpr (ATOMIC) {
      if (sum) atomicAdd(reinterpret_cast<unsigned long long*>(counts + blockIdx.y), (unsigned long long)sum);
    } else {
      counts[blockIdx.y] = (int64_t)sum;
    }
  }
}

// Workgroups per sample: one per per_block units of work, capped so the whole
// launch stays within about one residency round (cap workgroups in total).
unsigned per_sample_blocks(int64_t units, int64_t per_block, int B, int64_t cap) {
  const int64_t want = (units + per_block - 1) / per_block;
  return (unsigned)std::max<int64_t>(1, std::min(want, std::max<int64_t>(1, cap / B)));
}

}  // namespace

hipError_t launch_pack_occupancy(const float* logits, int B, int64_t n_voxels, uint32_t* bits, hipStream_t s) {
  const int64_t n_words = (n_voxels + 31) / 32;
  if (n_voxels % 4 == 0 && (uintptr_t)logits % 16 == 0) {
    const int64_t n_pass = (n_voxels / 4 + 64 * kChunks - 1) / (64 * kChunks);
    dim3 grid(per_sample_blocks(n_pass, 4, B, 2048), (unsigned)B);
    launch(k_pack_occupancy_vec, grid, dim3(256), 0, s, logits, n_voxels, n_words, bits);
  } else {
    const int64_t n_pass = (n_voxels + 64 * kGroups - 1) / (64 * kGroups);
    dim3 grid(per_sample_blocks(n_pass, 4, B, 2048), (unsigned)B);
    launch(k_pack_occupancy, grid, dim3(256), 0, s, logits, n_voxels, n_words, bits);
  }
  return hipGetLastError();
}

hipError_t launch_dynamic_voxels(const uint32_t* a, const uint32_t* b, int B, int64_t n_words, int64_t* counts,
                                 hipStream_t s) {
  const bool vec = (n_words % 4 == 0) && ((uintptr_t)a % 16 == 0) && ((uintptr_t)b % 16 == 0);
  // 32 words per thread and workgroup before splitting a sample (a 64^3 grid is one workgroup)
  dim3 grid(per_sample_blocks(n_words, 256 * 32, B, 2048), (unsigned)B);
  if (grid.x == 1) {
    if (vec)
      launch((k_dynamic_voxels<true, false>), grid, dim3(256), 0, s, a, b, n_words, counts);
    else
      launch((k_dynamic_voxels<false, false>), grid, dim3(256), 0, s, a, b, n_words, counts);
    return hipGetLastError();
  }
  launch(k_zero_counts, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, counts, B);
  if (vec)
    launch((k_dynamic_voxels<true, true>), grid, dim3(256), 0, s, a, b, n_words, counts);
  else
    launch((k_dynamic_voxels<false, true>), grid, dim3(256), 0, s, a, b, n_words, counts);
  return hipGetLastError();
}

}  // namespace f3c
