// Dense projections of the transformer blocks on the 32x32 matrix cores:
// C = A W^T + bias, A = activations [M][K] (row-major, K contiguous),
// W = weights [N][K] (torch Linear layout, K contiguous), f32 accumulation.
// Epilogues fuse the bias with a dtype store (QKV / cross-attention Q / KV),
// GELU (tanh form, MLP fc1), or a gated residual update in f32
// (h += gate * (.), attention output projections and MLP fc2).
//
// Workgroup tile BM x BN with 4 wavefronts in a 2 x 2 arrangement, each owning
// a (BM/2) x (BN/2) block of 32x32 MFMA accumulators. K is staged 128 bytes at
// a time through padded LDS rows (144-byte stride: the 16-byte fragment reads
// of 16 consecutive lanes cover all 64 banks once). The next K tile is fetched
// into registers while the current one is consumed, and written to the second
// LDS buffer, so one barrier per K tile suffices.
//
// The weight fragment is the MFMA's A operand and the activation fragment its
// B operand, i.e. each instruction produces a 32 x 32 tile of C^T: a lane then
// holds one activation row and four consecutive output columns per
// accumulator group, so the epilogue moves 8-byte (bf16) / 16-byte (f32)
// vectors. A lane reads 16 contiguous bytes of one row at K-group offset l/32
// for both operands; any common assignment of K elements to the instruction's
// K slots yields the same dot products.
#include <cmath>

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
  int xq;                             // column groups of the XCD tile partition (divides N / BN)
  float oscale;                       // stored outputs of columns < oscale_cols are multiplied by oscale
  int oscale_cols;
};

template <typename T>
__device__ __forceinline__ void store4(T* dst, const float (&v)[4]);
template <>
__device__ __forceinline__ void store4<float>(float* dst, const float (&v)[4]) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* dst, const float (&v)[4]) {
  bf16x4 o;
  o[0] = (bf16)v[0];
  o[1] = (bf16)v[1];
  o[2] = (bf16)v[2];
  o[3] = (bf16)v[3];
  *reinterpret_cast<bf16x4*>(dst) = o;
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, int EPI, int SITE, int PF = 1>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gemm(GemmArgs p) {
  constexpr int NT = 64 * WGM * WGN;                        // threads
  constexpr int WTM = BM / WGM, WTN = BN / WGN;             // wave tile
  constexpr int TM = WTM / 32, TN = WTN / 32;               // 32x32 tiles per wave
  constexpr int CA = BM * 8 / NT, CB = BN * 8 / NT;         // 16-byte chunks per thread
  constexpr int ES = sizeof(T);
  constexpr int PER16 = 16 / ES;                            // elements per 16 bytes
  constexpr int MMA_PER_READ = PER16 / Mfma<T>::E;          // instructions per fragment read
  constexpr int ABUF = BM * kRS, BBUF = BN * kRS;
  static_assert(CA >= 1 && CB >= 1 && TM >= 1 && TN >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) char lds[STAGES * (ABUF + BBUF)];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int g = lane >> 5, r32 = lane & 31;
  // Tile of this workgroup. Workgroups go round-robin to the 8 XCDs, each with
  // its own L2; the 1-D grid is remapped so that XCD j gets one contiguous run
  // of a tile order that is column-group major (xq groups of N/BN/xq column
  // tiles), then row-panel major. Each XCD then reads about 1/(8/xq) of A and
  // 1/xq of W instead of all of A (a row panel's column tiles on different
  // XCDs): HBM-side traffic xq*|A| + (8/xq)*|W|.
  int n0, m0;
  {
    const int gx = p.N / BN, gy = (p.M + BM - 1) / BM;
    const int l = xcd_logical_id(blockIdx.x, gx * gy);
    const int gq = gx / p.xq, per_group = gy * gq;
    const int grp = l / per_group, r = l - grp * per_group;
    const int y = r / gq;
    n0 = (grp * gq + (r - y * gq)) * BN;
    m0 = y * BM;
  }
  const size_t lda_b = (size_t)p.lda * ES, ldw_b = (size_t)p.ldw * ES;
  const int KT = (p.K * ES) / kBKB;
  constexpr size_t k_base = 0;

  // Rows past M are loaded from row M-1 (always valid) and never stored.
  const char* a_row[CA];
  const char* w_row[CB];
  int chunk_a[CA], chunk_b[CB];
#pragma unroll
  for (int q = 0; q < CA; ++q) {
    const int c = tid + NT * q, row = c >> 3;
    a_row[q] = p.A + (size_t)min(m0 + row, p.M - 1) * lda_b + k_base + (c & 7) * 16;
    chunk_a[q] = row * kRS + (c & 7) * 16;
  }
#pragma unroll
  for (int q = 0; q < CB; ++q) {
    const int c = tid + NT * q, row = c >> 3;
    w_row[q] = p.W + (size_t)(n0 + row) * ldw_b + k_base + (c & 7) * 16;
    chunk_b[q] = row * kRS + (c & 7) * 16;
  }

  // PF register sets: set r holds the tile whose index is congruent to r mod PF.
  u32x4 ra[PF][CA], rb[PF][CB];
  auto load_tile = [&](int kt, int r) {
    const size_t kb = (size_t)kt * kBKB;
#pragma unroll
    for (int q = 0; q < CA; ++q) ra[r][q] = *reinterpret_cast<const u32x4*>(a_row[q] + kb);
#pragma unroll
    for (int q = 0; q < CB; ++q) rb[r][q] = *reinterpret_cast<const u32x4*>(w_row[q] + kb);
  };
  auto store_tile = [&](int buf, int r) {
    char* As = lds + buf * (ABUF + BBUF);
    char* Bs = As + ABUF;
#pragma unroll
    for (int q = 0; q < CA; ++q) *reinterpret_cast<u32x4*>(As + chunk_a[q]) = ra[r][q];
#pragma unroll
    for (int q = 0; q < CB; ++q) *reinterpret_cast<u32x4*>(Bs + chunk_b[q]) = rb[r][q];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  auto compute = [&](int buf) {
    const char* As = lds + buf * (ABUF + BBUF);
    const char* Bs = As + ABUF;
#pragma unroll
    for (int ks = 0; ks < kBKB / 32; ++ks) {
      u32x4 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const u32x4*>(As + (wm * WTM + i * 32 + r32) * kRS + ks * 32 + g * 16);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const u32x4*>(Bs + (wn * WTN + j * 32 + r32) * kRS + ks * 32 + g * 16);
#pragma unroll
      for (int u = 0; u < MMA_PER_READ; ++u)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            typename Mfma<T>::frag a, w;
            if constexpr (sizeof(T) == 2) {
              a = __builtin_bit_cast(bf16x8, fa[i]);
              w = __builtin_bit_cast(bf16x8, fb[j]);
            } else {
              a = __builtin_bit_cast(f32x4, fa[i])[u];
              w = __builtin_bit_cast(f32x4, fb[j])[u];
            }
            acc[i][j] = Mfma<T>::mma(w, a, acc[i][j]);   // C^T tile: rows = output columns
          }
    }
  };

  if constexpr (PF == 1) {
    load_tile(0, 0);
    store_tile(0, 0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) load_tile(kt + 1, 0);
      if constexpr (STAGES == 2) {
        compute(kt & 1);
        if (kt + 1 < KT) store_tile((kt + 1) & 1, 0);
        __syncthreads();
      } else {
        compute(0);
        __syncthreads();
        if (kt + 1 < KT) {
          store_tile(0, 0);
          __syncthreads();
        }
      }
    }
  } else {
    // Prefetch distance PF (2 or 3) with double-buffered LDS: at step kt the
    // loads of tile kt+PF are issued while tile kt is consumed and tile kt+1
    // (loaded PF-1 steps earlier) is staged. Loads are issued unconditionally
    // (past the end they re-read the last tile), so the wait before staging
    // only covers the oldest load group.
    static_assert(STAGES == 2 && PF <= 3, "prefetch distance 2-3 needs two LDS buffers");
#pragma unroll
    for (int r = 0; r < PF; ++r) load_tile(min(r, KT - 1), r);
    store_tile(0, 0);
    __syncthreads();
    auto step = [&](int kt, int rr, int rl) {   // rr = kt % PF, rl = kt % 2 (constants below)
      load_tile(min(kt + PF, KT - 1), rr);
      // 64 x 64 tiles: keep the loads ahead of the compute. Scheduled after it
      // (to save registers) they leave nothing in flight when the older set is
      // staged, so the staging waits for every outstanding load (measured on
      // MI355X: fc2 at M = 820, 24.5 -> 20.9 us). The larger tiles are faster
      // with the compiler's own interleaving.
      if constexpr (BM == 64 && BN == 64) __builtin_amdgcn_sched_barrier(0);
      compute(rl);
      store_tile(rl ^ 1, rr + 1 == PF ? 0 : rr + 1);
      __syncthreads();
    };
    // Whole groups of U steps in the loop and the remainder after it, so the
    // loop's back edge is always taken after the last step of a group: the
    // register sets then have the same pending loads on every entry to the
    // loop head, and the compiler's waits there cover only the oldest group.
    constexpr int U = PF == 3 ? 6 : 2;
    int kt = 0;
    for (; kt + U <= KT; kt += U) {
#pragma unroll
      for (int i = 0; i < U; ++i) step(kt + i, i % PF, i & 1);
    }
#pragma unroll
    for (int i = 0; i < U - 1; ++i)
      if (kt + i < KT) step(kt + i, i % PF, i & 1);
  }

  // Epilogue. Tile (i, j), group q: activation row m0 + wm*BM/2 + 32 i + r32,
  // output columns n0 + wn*BN/2 + 32 j + 8 q + 4 g + (0..3).
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int row = m0 + wm * WTM + i * 32 + r32;
    if (row >= p.M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = n0 + wn * WTN + j * 32 + 8 * q + 4 * g;
        const float4 bv = *reinterpret_cast<const float4*>(p.bias + col);
        float v[4] = {acc[i][j][4 * q] + bv.x, acc[i][j][4 * q + 1] + bv.y, acc[i][j][4 * q + 2] + bv.z,
                      acc[i][j][4 * q + 3] + bv.w};
        if constexpr (EPI == EPI_RESID) {
          float4 gv = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
          if (p.gate) gv = *reinterpret_cast<const float4*>(p.gate + col);
          float4* r = reinterpret_cast<float4*>(p.resid + (size_t)row * p.ldr + col);
          float4 h = *r;
          h.x += gv.x * v[0];
          h.y += gv.y * v[1];
          h.z += gv.z * v[2];
          h.w += gv.w * v[3];
          *r = h;
        } else {
          if constexpr (EPI == EPI_GELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
          }
          if (col < p.oscale_cols) {        // four columns: all in or all out (oscale_cols % 4 == 0)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] *= p.oscale;
          }
          store4<T>(reinterpret_cast<T*>(p.out) + (size_t)row * p.ldo + col, v);
        }
      }
  }
}

// bf16 path. Workgroup tile BM x BN; every wave owns a 64 x 64 block (2 x 2
// accumulators of 32 x 32), so an MFMA costs 1 KiB of LDS reads (the
// 32 x 64-wave tiles above cost 1.5 KiB, more than the LDS delivers per
// MFMA). The NW waves are (BM/64)(BN/64) positions times KG K-groups: within
// every 64-element K tile, group kg takes the 16-element K-steps kg, kg + KG,
// ..., and at the end the groups' partial blocks are summed through LDS in
// group order (deterministic); each group then writes 4/KG of the block.
// K tiles go global -> LDS by DMA (no registers) into four buffers, three
// tiles ahead, one barrier per tile. LDS rows are the 128 bytes of a row's K
// tile with their 16-byte chunks XOR-swizzled by (row >> 1) & 7, which makes
// the fragment reads of 16 consecutive rows conflict-free.
template <int BM, int BN, int NW, int EPI, int SITE, int KTB = 128, int STAGES = 4, int DIST = 3>
__global__ __launch_bounds__(64 * NW) void k_gemm2(GemmArgs p) {
  constexpr int PM = BM / 64, PN = BN / 64, NPOS = PM * PN, KG = NW / NPOS;
  static_assert(NW % NPOS == 0 && (KG == 1 || KG == 2 || KG == 4), "waves must be positions x 1, 2 or 4");
  static_assert(KTB == 64 || KTB == 128, "K tile of 32 or 64 elements");
  static_assert((STAGES & (STAGES - 1)) == 0 && DIST < STAGES, "power-of-two stages, distance below");
  constexpr int CPR = KTB / 16;                         // 16-byte chunks per row
  constexpr int KSTEPS = KTB / 32 / KG;
  static_assert(KSTEPS >= 1, "each K-group needs a K-step per tile");
  constexpr int ABUF = BM * KTB, SBUF = (BM + BN) * KTB;
  constexpr int RPB = 1024 / KTB;                       // rows per 1 KiB DMA block
  constexpr int DA = BM / RPB, DB = BN / RPB;           // 1 KiB DMA blocks of a K tile
  constexpr int DQ = (DA + DB + NW - 1) / NW;           // blocks per wave
  constexpr int RED = NPOS * 4 * (KG - 1) * 4096;      // partial blocks exchanged at the end
  static_assert(RED <= STAGES * SBUF, "reduction must fit in the stage buffers");
  __shared__ __attribute__((aligned(16))) char lds[STAGES * SBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int pos = wave % NPOS, kg = wave / NPOS;
  const int wm = pos / PN, wn = pos % PN;
  const int g = lane >> 5, r32 = lane & 31;
  int n0, m0;
  {
    const int gx = p.N / BN, gy = (p.M + BM - 1) / BM;
    const int l = xcd_logical_id(blockIdx.x, gx * gy);
    const int gq = gx / p.xq, per_group = gy * gq;
    const int grp = l / per_group, r = l - grp * per_group;
    const int y = r / gq;
    n0 = (grp * gq + (r - y * gq)) * BN;
    m0 = y * BM;
  }
  const size_t lda_b = (size_t)p.lda * 2, ldw_b = (size_t)p.ldw * 2;
  const int KT = (p.K * 2) / KTB;
  constexpr size_t k_base = 0;

  // Swizzle of a row's 16-byte chunks: with 128-byte rows, (row >> 1) & 7;
  // with 64-byte rows, (row >> 2) & 3. Either way the fragment reads of 16
  // consecutive rows at one logical chunk hit all 64 banks once.
  auto swizzle = [](int row) { return KTB == 128 ? (row >> 1) & 7 : (row >> 2) & 3; };
  // DMA block b: A rows RPB*b.. (b < DA) or W rows RPB*(b - DA)..; lane l
  // fills row RPB*b + l/CPR at physical chunk l%CPR, i.e. loads the logical
  // chunk that the row's swizzle maps there. Rows past M re-read row M - 1
  // (never stored).
  const char* dsrc[DQ];
  int doff[DQ];
#pragma unroll
  for (int q = 0; q < DQ; ++q) {
    const int blk = min(wave + NW * q, DA + DB - 1);
    const int phys = lane % CPR;
    if (blk < DA) {
      const int row = RPB * blk + lane / CPR;
      dsrc[q] = p.A + (size_t)min(m0 + row, p.M - 1) * lda_b + k_base + ((phys ^ swizzle(row)) << 4);
      doff[q] = blk * 1024;
    } else {
      const int row = RPB * (blk - DA) + lane / CPR;
      dsrc[q] = p.W + (size_t)(n0 + row) * ldw_b + k_base + ((phys ^ swizzle(row)) << 4);
      doff[q] = ABUF + (blk - DA) * 1024;
    }
  }
  auto fetch = [&](int kt, int buf) {
#pragma unroll
    for (int q = 0; q < DQ; ++q) dma16(dsrc[q] + (size_t)kt * KTB, lds + buf * SBUF + doff[q]);
  };

  // Fragment reads: lane reads 16 bytes of row (block row + 32 i + r32) at
  // logical chunk 2 ks + g.
  const int swz = swizzle(r32);
  int chofs[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s) chofs[s] = ((2 * (kg + KG * s) + g) ^ swz) << 4;
  const int a_row = (wm * 64 + r32) * KTB, b_row = ABUF + (wn * 64 + r32) * KTB;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  auto compute = [&](int buf) {
    const char* base = lds + buf * SBUF;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = *reinterpret_cast<const u32x4*>(base + a_row + i * 32 * KTB + chofs[s]);
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[j] = *reinterpret_cast<const u32x4*>(base + b_row + j * 32 * KTB + chofs[s]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = Mfma<bf16>::mma(__builtin_bit_cast(bf16x8, fb[j]), __builtin_bit_cast(bf16x8, fa[i]), acc[i][j]);
    }
  };

  // Tile kt in buffer kt % STAGES. Iteration kt waits for tile kt (the next
  // DIST - 1 tiles stay in flight); the barrier makes every wave's DMA visible
  // and retires the buffer of tile kt - 1 (or older), which receives tile
  // kt + DIST (clamped: past the end the last tile is re-read, so the wait
  // count stays fixed).
#pragma unroll
  for (int r = 0; r < DIST; ++r) fetch(min(r, KT - 1), r);
  int buf = 0;
  for (int kt = 0; kt < KT; ++kt) {
    wait_vm<(DIST - 1) * DQ>();
    __syncthreads();
    fetch(min(kt + DIST, KT - 1), (buf + DIST) & (STAGES - 1));
    compute(buf);
    buf = (buf + 1) & (STAGES - 1);
  }
  wait_vm<0>();
  __syncthreads();                     // no DMA in flight, every wave past its last LDS read

  // Accumulator a = 2 i + j belongs to K-group a * KG / 4. The other groups
  // leave their partial in LDS (lane-major, 4 KiB per block); the owner adds
  // them in group order.
  auto owner = [](int a) { return a * KG / 4; };
  if constexpr (KG > 1) {
    float* red = reinterpret_cast<float*>(lds);
    auto slot = [&](int a, int k) {      // k != owner(a)
      const int kk = k < owner(a) ? k : k - 1;
      return red + (((size_t)pos * 4 + a) * (KG - 1) + kk) * 1024;
    };
#pragma unroll
    for (int a = 0; a < 4; ++a)
      if (owner(a) != kg) {
        float* dst = slot(a, kg);
#pragma unroll
        for (int e = 0; e < 16; ++e) dst[e * 64 + lane] = acc[a >> 1][a & 1][e];
      }
    __syncthreads();
#pragma unroll
    for (int a = 0; a < 4; ++a)
      if (owner(a) == kg) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float sum = 0.0f;
#pragma unroll
          for (int k = 0; k < KG; ++k) sum += (k == kg) ? acc[a >> 1][a & 1][e] : slot(a, k)[e * 64 + lane];
          acc[a >> 1][a & 1][e] = sum;
        }
      }
  }

  // Epilogue of the owned blocks. Block (i, j), group q: activation row
  // m0 + 64 wm + 32 i + r32, output columns n0 + 64 wn + 32 j + 8 q + 4 g + (0..3).
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    if (owner(a) != kg) continue;
    const int i = a >> 1, j = a & 1;
    const int row = m0 + wm * 64 + i * 32 + r32;
    if (row >= p.M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = n0 + wn * 64 + j * 32 + 8 * q + 4 * g;
      const f32x16& c = acc[i][j];
      const float4 bv = *reinterpret_cast<const float4*>(p.bias + col);
      float v[4] = {c[4 * q] + bv.x, c[4 * q + 1] + bv.y, c[4 * q + 2] + bv.z, c[4 * q + 3] + bv.w};
      if constexpr (EPI == EPI_RESID) {
        float4 gv = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
        if (p.gate) gv = *reinterpret_cast<const float4*>(p.gate + col);
        float4* r = reinterpret_cast<float4*>(p.resid + (size_t)row * p.ldr + col);
        float4 h = *r;
        h.x += gv.x * v[0];
        h.y += gv.y * v[1];
        h.z += gv.z * v[2];
        h.w += gv.w * v[3];
        *r = h;
      } else {
        if constexpr (EPI == EPI_GELU) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
        }
        if (col < p.oscale_cols) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= p.oscale;
        }
        store4<bf16>(reinterpret_cast<bf16*>(p.out) + (size_t)row * p.ldo + col, v);
      }
    }
  }
}

// Large projections (tens of thousands of rows): 256 x 256 tiles of 8 waves,
// each owning a 128 x 64 block (4 x 2 accumulators of 32 x 32), two waves per
// SIMD. K tiles of 64 elements go HBM -> LDS by DMA into two stages (XOR
// swizzled 128-byte rows as in k_gemm2). Each 16-element K-step is one
// inline-assembly block: it waits for its own fragments, then interleaves the
// six fragment reads of the next K-step with its eight MFMAs, so LDS latency
// stays behind matrix work without depending on the compiler's schedule.
// Before the last K-step of a tile every wave holds that step's fragments, so
// one barrier (after the DMA of the next tile landed) retires the tile's
// stage, which then receives the tile after next, and makes the next tile
// readable: the last K-step already reads the next tile's first fragments.
// Same K order and instruction as k_gemm, so its results are bit-identical.
// Requires N % 256 == 0 and K % 128 == 0 (an even number of K tiles).
// K-step with prefetch: acc[i][j] += W[j] A[i] (i < 4, j < 2), and the six
// fragments of the next K-step read into the other register set.
#define G3_STEP_PF(C, FA, FW, NA, NW, AAD, WAD)                                                                \
  asm volatile("s_waitcnt lgkmcnt(0)\n\t"                                                                      \
               "ds_read_b128 %[na0], %[aad]\n\t"                                                               \
               "v_mfma_f32_32x32x16_bf16 %[c00], %[w0], %[a0], %[c00]\n\t"                                     \
               "ds_read_b128 %[na1], %[aad] offset:4096\n\t"                                                   \
               "v_mfma_f32_32x32x16_bf16 %[c01], %[w1], %[a0], %[c01]\n\t"                                     \
               "ds_read_b128 %[na2], %[aad] offset:8192\n\t"                                                   \
               "v_mfma_f32_32x32x16_bf16 %[c10], %[w0], %[a1], %[c10]\n\t"                                     \
               "ds_read_b128 %[na3], %[aad] offset:12288\n\t"                                                  \
               "v_mfma_f32_32x32x16_bf16 %[c11], %[w1], %[a1], %[c11]\n\t"                                     \
               "ds_read_b128 %[nw0], %[wad]\n\t"                                                               \
               "v_mfma_f32_32x32x16_bf16 %[c20], %[w0], %[a2], %[c20]\n\t"                                     \
               "ds_read_b128 %[nw1], %[wad] offset:4096\n\t"                                                   \
               "v_mfma_f32_32x32x16_bf16 %[c21], %[w1], %[a2], %[c21]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c30], %[w0], %[a3], %[c30]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c31], %[w1], %[a3], %[c31]"                                         \
               : [c00] "+v"(C[0][0]), [c01] "+v"(C[0][1]), [c10] "+v"(C[1][0]), [c11] "+v"(C[1][1]),            \
                 [c20] "+v"(C[2][0]), [c21] "+v"(C[2][1]), [c30] "+v"(C[3][0]), [c31] "+v"(C[3][1]),            \
                 [na0] "=&v"(NA[0]), [na1] "=&v"(NA[1]), [na2] "=&v"(NA[2]), [na3] "=&v"(NA[3]),               \
                 [nw0] "=&v"(NW[0]), [nw1] "=&v"(NW[1])                                                        \
               : [a0] "v"(FA[0]), [a1] "v"(FA[1]), [a2] "v"(FA[2]), [a3] "v"(FA[3]), [w0] "v"(FW[0]),          \
                 [w1] "v"(FW[1]), [aad] "v"(AAD), [wad] "v"(WAD))

#define G3_STEP(C, FA, FW)                                                                                     \
  asm volatile("s_waitcnt lgkmcnt(0)\n\t"                                                                      \
               "v_mfma_f32_32x32x16_bf16 %[c00], %[w0], %[a0], %[c00]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c01], %[w1], %[a0], %[c01]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c10], %[w0], %[a1], %[c10]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c11], %[w1], %[a1], %[c11]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c20], %[w0], %[a2], %[c20]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c21], %[w1], %[a2], %[c21]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c30], %[w0], %[a3], %[c30]\n\t"                                     \
               "v_mfma_f32_32x32x16_bf16 %[c31], %[w1], %[a3], %[c31]"                                         \
               : [c00] "+v"(C[0][0]), [c01] "+v"(C[0][1]), [c10] "+v"(C[1][0]), [c11] "+v"(C[1][1]),            \
                 [c20] "+v"(C[2][0]), [c21] "+v"(C[2][1]), [c30] "+v"(C[3][0]), [c31] "+v"(C[3][1])             \
               : [a0] "v"(FA[0]), [a1] "v"(FA[1]), [a2] "v"(FA[2]), [a3] "v"(FA[3]), [w0] "v"(FW[0]),          \
                 [w1] "v"(FW[1]))

template <int EPI, int SITE>
__global__ __launch_bounds__(512) void k_gemm_big(GemmArgs p) {
  constexpr int BM = 256, BN = 256, KTB = 128, SBUF = (BM + BN) * KTB, ABUF = BM * KTB;
  __shared__ __attribute__((aligned(16))) char lds[2 * SBUF];   // 128 KiB
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;                      // 128-row half, 64-column quarter
  const int g = lane >> 5, r32 = lane & 31;
  int n0, m0;
  {
    const int gx = p.N / BN, gy = (p.M + BM - 1) / BM;
    const int l = xcd_logical_id(blockIdx.x, gx * gy);
    const int gq = gx / p.xq, per_group = gy * gq;
    const int grp = l / per_group, r = l - grp * per_group;
    const int y = r / gq;
    n0 = (grp * gq + (r - y * gq)) * BN;
    m0 = y * BM;
  }
  const size_t lda_b = (size_t)p.lda * 2, ldw_b = (size_t)p.ldw * 2;
  const int KT = (p.K * 2) / KTB;
  // DMA: 64 blocks of 1 KiB (8 rows of 128 bytes) per tile: A rows 8b.. for
  // b < 32, W rows 8(b-32).. for b >= 32; wave w takes blocks w, w+8, ...
  // Lane l fills row 8b + l/8 at physical chunk l%8 with the logical chunk the
  // row's swizzle ((row >> 1) & 7) maps there.
  const char* dsrc[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int blk = wave + 8 * q;
    const int phys = lane & 7, rr = lane >> 3;
    if (blk < 32) {
      const int row = 8 * blk + rr;
      dsrc[q] = p.A + (size_t)min(m0 + row, p.M - 1) * lda_b + ((phys ^ ((row >> 1) & 7)) << 4);
    } else {
      const int row = 8 * (blk - 32) + rr;
      dsrc[q] = p.W + (size_t)(n0 + row) * ldw_b + ((phys ^ ((row >> 1) & 7)) << 4);
    }
  }
  auto fetch = [&](int kt, int stage) {
#pragma unroll
    for (int q = 0; q < 8; ++q) dma16(dsrc[q] + (size_t)kt * KTB, lds + stage * SBUF + (wave + 8 * q) * 1024);
  };
  // Fragment read bases (bytes): A row wm*128 + r32, W row wn*64 + r32, logical
  // chunk 2ks + g -> physical (2ks + g) ^ ((r32 >> 1) & 7).
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const int swz = (r32 >> 1) & 7;
  uint32_t aad[2][4], wad[2][4];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint32_t ch = (uint32_t)(((2 * ks + g) ^ swz) << 4);
      aad[s][ks] = lds0 + s * SBUF + (wm * 128 + r32) * KTB + ch;
      wad[s][ks] = lds0 + s * SBUF + ABUF + (wn * 64 + r32) * KTB + ch;
    }
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  u32x4 fa[2][4], fw[2][2];
  auto read_frags = [&](int s) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(fa[0][i]) : "v"(aad[s][0]), "i"(i * 4096));
#pragma unroll
    for (int j = 0; j < 2; ++j)
      asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(fw[0][j]) : "v"(wad[s][0]), "i"(j * 4096));
  };
  // Tile kt in stage s: K-step ks uses register set ks & 1 and reads the next
  // step's fragments into the other set. Before the last K-step every wave
  // holds that step's fragments, so one barrier (after the DMA of tile kt + 1
  // landed) both retires stage s, which then receives tile kt + 2, and makes
  // stage s ^ 1 readable: the last K-step reads the first fragments of tile
  // kt + 1 while its MFMAs run.
  auto tile = [&](int kt, int s) {
    G3_STEP_PF(acc, fa[0], fw[0], fa[1], fw[1], aad[s][1], wad[s][1]);
    G3_STEP_PF(acc, fa[1], fw[1], fa[0], fw[0], aad[s][2], wad[s][2]);
    G3_STEP_PF(acc, fa[0], fw[0], fa[1], fw[1], aad[s][3], wad[s][3]);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wait_vm<0>();
    __syncthreads();
    fetch(min(kt + 2, KT - 1), s);
    G3_STEP_PF(acc, fa[1], fw[1], fa[0], fw[0], aad[s ^ 1][0], wad[s ^ 1][0]);
  };
  // KT is even (K a multiple of 128).
  fetch(0, 0);
  wait_vm<0>();
  __syncthreads();
  read_frags(0);
  fetch(min(1, KT - 1), 1);
  for (int kt = 0; kt < KT; kt += 2) {
    tile(kt, 0);
    tile(kt + 1, 1);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  wait_vm<0>();
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");   // MFMA results before the reads below

  // Epilogue: block (i, j) of this wave, group q: activation row
  // m0 + 128 wm + 32 i + r32, output columns n0 + 64 wn + 32 j + 8 q + 4 g + (0..3).
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + wm * 128 + i * 32 + r32;
    if (row >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = n0 + wn * 64 + j * 32 + 8 * q + 4 * g;
        const f32x16& c = acc[i][j];
        const float4 bv = *reinterpret_cast<const float4*>(p.bias + col);
        float v[4] = {c[4 * q] + bv.x, c[4 * q + 1] + bv.y, c[4 * q + 2] + bv.z, c[4 * q + 3] + bv.w};
        if constexpr (EPI == EPI_RESID) {
          float4 gv = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
          if (p.gate) gv = *reinterpret_cast<const float4*>(p.gate + col);
          float4* r = reinterpret_cast<float4*>(p.resid + (size_t)row * p.ldr + col);
          float4 h = *r;
          h.x += gv.x * v[0];
          h.y += gv.y * v[1];
          h.z += gv.z * v[2];
          h.w += gv.w * v[3];
          *r = h;
        } else {
          if constexpr (EPI == EPI_GELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
          }
          if (col < p.oscale_cols) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] *= p.oscale;
          }
          store4<bf16>(reinterpret_cast<bf16*>(p.out) + (size_t)row * p.ldo + col, v);
        }
      }
  }
}


template <int BM, int BN, int NW, int EPI, int SITE, int KTB = 128, int STAGES = 4, int DIST = 3>
hipError_t launch_cfg2(const GemmArgs& a, hipStream_t s) {
  if (a.xq < 1 || (a.N / BN) % a.xq) return hipErrorInvalidValue;
  dim3 grid((a.N / BN) * ((a.M + BM - 1) / BM));
  launch((k_gemm2<BM, BN, NW, EPI, SITE, KTB, STAGES, DIST>), grid, dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

template <typename T, int BM, int BN, int WGM, int WGN, int STAGES, int EPI, int SITE, int PF = 1>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  if (a.xq < 1 || (a.N / BN) % a.xq) return hipErrorInvalidValue;
  dim3 grid((a.N / BN) * ((a.M + BM - 1) / BM));
  launch((k_gemm<T, BM, BN, WGM, WGN, STAGES, EPI, SITE, PF>), grid, dim3(64 * WGM * WGN), 0, s, a);
  return hipGetLastError();
}

// Tile choice for the register-staged bf16 kernel: the smallest estimated
// time over 128 x 128 (8 waves), 64 x 128 and 64 x 64 (4 waves) tiles. Model
// per tile shape: a fixed cost plus, per 1024 of K, a cost per round of 256
// workgroups (a partial round costs a whole one) and a smaller cost per
// workgroup (L2 and HBM contention); least-squares fit to 52 measurements on
// MI355X with random bf16 operands at M = 820 ... 4055, N = 1024 / 3072 /
// 4096, K = 1024 / 4096 (rms 1.1 / 1.8 / 1.1 us). Over those shapes it picks
// within 0.2% of the best tile in total time (the earlier rounds-only model:
// 1.4%, up to 11% on single shapes).
inline int choose_tiles(int M, int N, int K) {
  struct Cost { int bm, bn; double fixed, per_round, per_load; };
  constexpr Cost kCost[3] = {{128, 128, 6.37, 6.73, 2.86}, {64, 128, 6.16, 4.85, 1.10}, {64, 64, 5.35, 2.51, 0.85}};
  int cfg = 0;
  double best = 0.0;
  for (int c = 0; c < 3; ++c) {
    const double load = (double)((M + kCost[c].bm - 1) / kCost[c].bm) * (N / kCost[c].bn) / 256.0;
    const double t = kCost[c].fixed + K / 1024.0 * (kCost[c].per_round * std::ceil(load) + kCost[c].per_load * load);
    if (c == 0 || t < best) {
      best = t;
      cfg = c;
    }
  }
  return cfg;
}

// Column groups of the XCD tile partition (see k_gemm): over the 8 XCDs, A is
// read xq times and W 8/xq times in all.
// Pick the xq (dividing the column-tile count) that minimises that traffic
// while one XCD's share of W (|W|/xq) stays within half of its 4 MiB L2, so
// the row panels that follow each other on an XCD find it resident. Measured
// on MI355X against the plain 2-D grid: fc2 at M = 4096, 46.6 -> 39.6 us;
// o at M = 4096, 19.0 -> 17.8 us; QKV and fc1 unchanged.
inline int choose_xq(int M, int N, int K, int es, int BN) {
  const int gx = N / BN;
  const double a = (double)M * K * es, w = (double)N * K * es, l2_share = 2.0 * 1024 * 1024;
  int best = 1;
  double best_cost = 0.0;
  bool best_fits = false;
  for (int q = 1; q <= 8; q *= 2) {
    if (gx % q) continue;
    const bool fits = w / q <= l2_share;
    const double cost = a * q + w * (8.0 / q);
    if (q == 1 || (fits && !best_fits) || (fits == best_fits && cost <= best_cost)) {
      best = q;
      best_cost = cost;
      best_fits = fits;
    }
  }
  return best;
}

// bf16: long K (>= 4096, the MLP's second projection) that fits one round of
// 64 x 64 or 64 x 128 workgroups goes to k_gemm2 with four K-groups per
// position (measured on MI355X at N = 1024, K = 4096: M = 820, 17.5 us against
// 20.6 us for the best staged tile; M = 1310 ... 1915, 24.4 against 29.3 us);
// everything else to the register-staged kernel.
template <int EPI, int SITE>
hipError_t launch_big(const GemmArgs& a, hipStream_t s) {
  if (a.xq < 1 || (a.N / 256) % a.xq) return hipErrorInvalidValue;
  launch((k_gemm_big<EPI, SITE>), dim3((a.N / 256) * ((a.M + 255) / 256)), dim3(512), 0, s, a);
  return hipGetLastError();
}

// Where the 256 x 256 kernel wins inside the sampler (MI355X, against the
// 128 x 128 tiles): from 8192 rows, the QKV projection (N = 3K; 32768 rows:
// 270 -> 231 us, 9831 rows: 90 -> 78 us in the sampler's traces), the MLP's
// first projection (N = 4K, GELU; 32768 rows: 451-457 -> 386 us, 9831 rows:
// 127-129 -> 121 us) and its second (K = 4096; 339 against 418-437 us at 32768
// rows). The 1024-wide K = 1024 projections stay on 128 x 128 tiles (a tie at
// 32768 rows, 50 against 45 us at 9831): one 128 KiB workgroup per CU cannot
// hide its residual epilogue behind another workgroup's main loop.
inline bool use_big(int M, int N, int K) {
  if (N % 256 || K % 128 || M < 8192) return false;
  return N == 3 * K || N == 4 * K || K >= 4096;
}

// Column groups of the 256 x 256 kernel. With K = 4096 the weight (8 MiB at
// N = 1024) cannot stay in an XCD's L2 whatever the grouping, while the four
// column tiles of a row panel run side by side on one XCD and share its
// 2 MiB A panel; so each XCD takes whole row panels (xq = 1: A read once;
// 32768 rows 339 us against 363 us at xq = 4, the L2-fit rule's pick). The
// GELU projection (N = 4K) measured best at two column groups (32768 rows:
// 386 against 407-410 us at xq = 4; 9831 rows: 121 against 125-128 us).
inline int big_xq(int M, int N, int K) {
  if (K >= 4096) return 1;
  if (N == 4 * K && (N / 256) % 2 == 0) return 2;
  return choose_xq(M, N, K, 2, 256);
}

template <typename T, int EPI, int SITE>
hipError_t launch_t(const GemmArgs& a0, hipStream_t s) {
  GemmArgs a = a0;
  if constexpr (sizeof(T) == 2) {
    if (use_big(a.M, a.N, a.K)) {
      a.xq = big_xq(a.M, a.N, a.K);
      return launch_big<EPI, SITE>(a, s);
    }
    const long rows64 = (a.M + 63) / 64;
    if (a.K >= 4096 && rows64 * (a.N / 64) <= 256) {
      a.xq = choose_xq(a.M, a.N, a.K, 2, 64);
      return launch_cfg2<64, 64, 4, EPI, SITE>(a, s);
    }
    if (a.K >= 4096 && rows64 * (a.N / 128) <= 256) {
      a.xq = choose_xq(a.M, a.N, a.K, 2, 128);
      return launch_cfg2<64, 128, 8, EPI, SITE>(a, s);
    }
    const int cfg = choose_tiles(a.M, a.N, a.K);
    a.xq = choose_xq(a.M, a.N, a.K, 2, cfg == 2 ? 64 : 128);
    if (cfg == 0) return launch_cfg<T, 128, 128, 2, 4, 2, EPI, SITE, 2>(a, s);
    if (cfg == 1) return launch_cfg<T, 64, 128, 2, 2, 2, EPI, SITE, 2>(a, s);
    return launch_cfg<T, 64, 64, 2, 2, 2, EPI, SITE, 2>(a, s);
  } else {
    a.xq = choose_xq(a.M, a.N, a.K, sizeof(T), 128);
    return launch_cfg<T, 64, 128, 2, 2, 2, EPI, SITE, 2>(a, s);
  }
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
                       hipStream_t s, float oscale, int oscale_cols) {
  if (M == 0) return hipSuccess;
  if (oscale_cols % 4) return hipErrorInvalidValue;
  GemmArgs a{M, N, K, (const char*)A, lda, (const char*)W, ldw, bias, gate, out, ldo, resid, ldr, 1, oscale,
             oscale_cols};
  return dt == DT_BF16 ? launch_site<bf16>(site, epi, a, s) : launch_site<float>(site, epi, a, s);
}

}  // namespace f3c
