// Variable-length multi-head softmax attention on the 32x32 matrix cores, used
// for self-attention over the active tokens of each sample (Sec. 4.2: self
// attention runs on the active subset only) and for cross-attention from the
// active tokens to the image-condition tokens.
//
// Online softmax over key/value tiles of 64 staged in LDS (V stored
// transposed). Each wavefront owns 32 queries and computes S^T = K Q^T, so a
// lane holds one query's scores for 16 of every 32 keys: the running max and
// sum are per-lane values combined with a single cross-half exchange
// (lane l with l ^ 32). The same accumulator layout feeds O^T = V^T P^T as the
// B operand without any data movement; the K-slot order of P (keys
// 8*(e/4) + 4*(l/32) + e%4) is matched when the V^T fragment is read.
//
// Scores on the matrix-core path (bf16, 64-wide heads) come out of the MFMAs
// already shifted: each score tile's accumulation starts from -m (the
// reference max), so a probability costs one exponential (and, unless the
// queries were stored multiplied by log2(e)/sqrt(hd), one multiply) plus its
// bf16 conversion.
//
// Pipelining. bf16 with 64-wide heads (the transformer's case): K and V tiles
// go from global memory straight into five LDS buffers (four with key groups)
// with 16-byte DMA loads issued three tiles ahead (two with key groups), and
// the score product of tile t+1 is issued before the softmax and PV product of
// tile t, so the matrix cores have independent work while the vector unit runs
// the softmax. Other types and head sizes
// fetch the next tile into registers while the current one is consumed and
// write it to the other of two LDS buffers. One barrier per tile either way.
// Only the last, ragged tile is masked. The running max is updated lazily:
// the accumulators are rescaled only when some query's max grows by more than
// 2^8 (in base-2 units), which keeps every unnormalised probability below 2^8
// and the result unchanged up to rounding.
//
// Few query tiles (late cached steps: a few hundred active tokens) cannot fill
// 256 CUs, so the key range may be split: each split writes its unnormalised
// output with its reference max and sum in f32, and a second kernel merges the
// splits in split order (the standard log-sum-exp combination; deterministic).
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace f3c {

namespace {

constexpr int kBKV = 64;             // keys per LDS tile

// max(a, b, c) as one v_max3_f32. fmaxf on MFMA results costs three
// instructions each (both inputs are first quieted with v_max x, x, since the
// compiler cannot prove they are not signalling NaNs); the scores here are
// finite or -inf, never NaN.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Max of the 16 accumulators of one 32 x 32 score tile: eight dependent
// v_max3_f32 in one block (one hazard boundary for the compiler instead of
// one per instruction; dependent VALU instructions need no wait states).
__device__ __forceinline__ float max16(const f32x16& v) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3\n\t"
      "v_max3_f32 %0, %0, %4, %5\n\t"
      "v_max3_f32 %0, %0, %6, %7\n\t"
      "v_max3_f32 %0, %0, %8, %9\n\t"
      "v_max3_f32 %0, %0, %10, %11\n\t"
      "v_max3_f32 %0, %0, %12, %13\n\t"
      "v_max3_f32 %0, %0, %14, %15\n\t"
      "v_max_f32 %0, %0, %16"
      : "=&v"(r)
      : "v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3]), "v"(v[4]), "v"(v[5]), "v"(v[6]), "v"(v[7]), "v"(v[8]),
        "v"(v[9]), "v"(v[10]), "v"(v[11]), "v"(v[12]), "v"(v[13]), "v"(v[14]), "v"(v[15]));
  return r;
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
constexpr float kRescaleLog2 = 8.0f;
// DMA path: a tile's probabilities are taken against the running reference
// max; when a lane's 32 probabilities sum to more than this, the reference is
// moved to the tile's max and the tile recomputed (so every probability that
// enters the PV product is at most 2^16).
constexpr float kTileSumLimit = 65536.0f;

struct AttnArgs {
  Segs qs, ks;
  int tile_off[kMaxBatch + 1];   // prefix of query tiles per sample
  const char* q;
  const char* k;
  const char* v;
  char* o;
  int ldq, ldk, ldv, ldo;        // elements
  int heads;
  float scale_log2;              // log2(e) / sqrt(hd), or 1 when the queries were stored scaled by it
  int splits;                    // key-range splits (1: normalised output straight to o)
  int rows;                      // query rows qs.off[B] - qs.off[0] (split partials)
  float* part_o;                 // [splits][rows][heads][hd] unnormalised outputs
  float* part_ml;                // [splits][rows][heads][2] (max * scale_log2, sum)
};

// KS key groups (matrix-core path only): the NW waves are NW/KS query waves
// times KS groups; group k takes key tiles t_begin + KS*i + k in lockstep
// with the others (one LDS stage holds the KS tiles of a step), and the
// groups' (max, sum, output) are merged through LDS at the end. Two groups
// double the waves per query tile where query tiles are too few to fill the
// chip.
// QS: the queries were stored multiplied by log2(e)/sqrt(hd) (scores come out
// in base-2 units).
template <typename T, int HD, int NW, int SITE, bool SPLIT, int KS = 1, bool QS = false>
__global__ __launch_bounds__(64 * NW) void k_attn(AttnArgs p) {
  constexpr int NT = 64 * NW;
  constexpr int QW = NW / KS;                // query waves
  constexpr int BQ = 32 * QW;
  constexpr int ES = sizeof(T);
  constexpr int E = Mfma<T>::E;
  // bf16 with 64-wide heads: K and V tiles go global -> LDS directly (16-byte
  // DMA loads, no registers) into five buffers (four with key groups), row-major
  // with 128-byte rows
  // whose 16-byte chunks are XOR-swizzled by row (conflict-free fragment
  // reads); V^T fragments come from the row-major V tile through the LDS
  // transpose read. Other types and head sizes stage through registers, with
  // V transposed on its way into LDS.
  constexpr bool DMA = ES == 2 && HD == 64;
  static_assert(KS == 1 || (KS == 2 && DMA && NW % 2 == 0 && !SPLIT),
                "key groups need the matrix-core path and the whole key range");
  constexpr int NBUF = DMA ? (KS == 1 ? 5 : 4) : 2;
  constexpr int KRS = DMA ? HD * ES : HD * ES + 16;   // K tile row stride (bytes)
  constexpr int VRS = kBKV * ES + 8;                 // V^T tile row stride (bytes), register path
  constexpr int NKS = HD * ES / 32;          // 32-byte K slices over the head dim
  constexpr int PER16 = 16 / ES;
  constexpr int MMA_PER_READ = PER16 / E;
  constexpr int HT = HD / 32;                // 32-row output tiles over the head dim
  constexpr int CPR = HD * ES / 16;          // 16-byte chunks per key row
  constexpr int KITEMS = kBKV * CPR;        // K chunks per tile
  constexpr int VITEMS = kBKV / 2 * CPR;    // V (key pair, chunk) items per tile
  constexpr int KCH = (KITEMS + NT - 1) / NT;
  constexpr int VPR = (VITEMS + NT - 1) / NT;
  constexpr int KBUF = kBKV * KRS, VBUF = DMA ? kBKV * HD * ES : HD * VRS;
  constexpr int TB = KBUF + VBUF, SB = KS * TB;      // bytes per tile, per stage
  // DMA path: the K tiles of all stages, then the V tiles (VREG on), so that a
  // fragment read's stage offset fits the 16-bit offset field of the LDS read.
  constexpr int VREG = NBUF * KS * KBUF;
  __shared__ __attribute__((aligned(16))) char lds[NBUF * SB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kgrp = wave / QW, qw = wave - kgrp * QW;
  const int g = lane >> 5, r32 = lane & 31;
  // 1-D grid over (head, query tile, split); all work of a head shares one XCD's L2.
  const int ntq = p.tile_off[p.qs.B];
  const int nsp = SPLIT ? p.splits : 1;
  const int logical = xcd_logical_id(blockIdx.x, ntq * p.heads * nsp);
  const int head = logical / (ntq * nsp);
  const int rem = logical - head * ntq * nsp;
  const int tq = rem / nsp, sp = rem - tq * nsp;
  const int b = find_segment(p.tile_off, p.qs.B, tq);
  const int qt = tq - p.tile_off[b];
  const int q_begin = p.qs.off[b], nq = p.qs.off[b + 1] - q_begin;
  const int k_begin = p.ks.off[b], nk = p.ks.off[b + 1] - k_begin;
  const int qi = qt * BQ + qw * 32 + r32;              // query of this lane (within the sample)
  const bool q_ok = qi < nq;

  // Q^T as the B operand: lane reads 16 bytes of its query row per 32-byte slice.
  u32x4 qf[NKS];
  {
    const char* qrow = p.q + ((size_t)(q_begin + (q_ok ? qi : 0)) * p.ldq + head * HD) * ES;
#pragma unroll
    for (int s = 0; s < NKS; ++s)
      qf[s] = q_ok ? *reinterpret_cast<const u32x4*>(qrow + s * 32 + g * 16) : u32x4{0, 0, 0, 0};
  }

  // Tile staging: K row-major, V transposed (pairs of keys per 32/64-bit write).
  // Keys past the end are read from the last key (always valid) and masked.
  // Two register sets: tile t+2 is fetched while tile t+1 waits to be staged.
  // Every thread issues the same loads (threads past the item count re-read
  // the last item and skip the LDS write): a branch around some of the loads
  // would make the compiler's wait before staging cover the loads in flight.
  u32x4 rk[2][KCH], rv[2][VPR][2];
  auto fetch = [&](int kv0, int r) {
#pragma unroll
    for (int q = 0; q < KCH; ++q) {
      const int ch = min(tid + NT * q, KITEMS - 1), row = ch / CPR, col = ch % CPR;
      const int key = min(kv0 + row, nk - 1);
      rk[r][q] = *reinterpret_cast<const u32x4*>(p.k + ((size_t)(k_begin + key) * p.ldk + head * HD) * ES + col * 16);
    }
#pragma unroll
    for (int q = 0; q < VPR; ++q) {
      const int it = min(tid + NT * q, VITEMS - 1), pr = it / CPR, col = it % CPR;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int key = min(kv0 + 2 * pr + h, nk - 1);
        rv[r][q][h] = *reinterpret_cast<const u32x4*>(p.v + ((size_t)(k_begin + key) * p.ldv + head * HD) * ES + col * 16);
      }
    }
  };
  auto stage = [&](int buf, int r) {
    char* Ks = lds + buf * (KBUF + VBUF);
    char* Vt = Ks + KBUF;
#pragma unroll
    for (int q = 0; q < KCH; ++q) {
      const int ch = tid + NT * q, row = ch / CPR, col = ch % CPR;
      if (KITEMS % NT != 0 && ch >= KITEMS) break;
      *reinterpret_cast<u32x4*>(Ks + row * KRS + col * 16) = rk[r][q];
    }
#pragma unroll
    for (int q = 0; q < VPR; ++q) {
      const int it = tid + NT * q, pr = it / CPR, col = it % CPR;
      if (VITEMS % NT != 0 && it >= VITEMS) break;
      const T* v0 = reinterpret_cast<const T*>(&rv[r][q][0]);
      const T* v1 = reinterpret_cast<const T*>(&rv[r][q][1]);
#pragma unroll
      for (int e = 0; e < PER16; ++e) {
        char* dst = Vt + (col * PER16 + e) * VRS + 2 * pr * ES;
        if constexpr (ES == 2) {
          const uint32_t lo = __builtin_bit_cast(uint16_t, v0[e]), hi = __builtin_bit_cast(uint16_t, v1[e]);
          *reinterpret_cast<uint32_t*>(dst) = lo | (hi << 16);
        } else {
          *reinterpret_cast<float2*>(dst) = make_float2(v0[e], v1[e]);
        }
      }
    }
  };

  // DMA path: one wave instruction fills 1 KiB = 8 rows; lane l writes 16-byte
  // slot l, i.e. row l/8 and physical chunk l%8, with the logical chunk the
  // row's swizzle maps there (XOR is its own inverse).
  //   K: physical chunk = chunk ^ ((row >> 1) & 7)  (16 lanes read 16 rows)
  //   V: physical chunk = chunk ^ (((row >> 1) & 1) << 2)  (transpose reads
  //      take 32 bytes from each of 4 consecutive rows)
  constexpr int DBLK = kBKV / 8;                       // 8-row blocks per tile
  constexpr int DQ = (DBLK + NW - 1) / NW;             // blocks per wave
  // DMA addresses: scalar bases (this sample's first key row of this head) and
  // 32-bit lane offsets, the same for every tile but for the key index (the
  // host checks that nk rows of either operand stay below 2 GiB); M0 from
  // wave-uniform values. Four vector instructions per tile instead of ten.
  const char* kbase = p.k + ((size_t)k_begin * p.ldk + head * HD) * ES;
  const char* vbase = p.v + ((size_t)k_begin * p.ldv + head * HD) * ES;
  const uint32_t ldk_b = (uint32_t)p.ldk * ES, ldv_b = (uint32_t)p.ldv * ES;
  const uint32_t lds_u = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto fetch_dma = [&](int kv0, int stage, int k) {
#pragma unroll
    for (int q = 0; q < DQ; ++q) {
      const int blk_u = min(wave_u + NW * q, DBLK - 1);
      const int row = blk_u * 8 + (lane >> 3), phys = lane & 7;
      const uint32_t key = (uint32_t)min(kv0 + row, nk - 1);
      const uint32_t kofs = key * ldk_b + (uint32_t)((phys ^ ((row >> 1) & 7)) << 4);
      const uint32_t vofs = key * ldv_b + (uint32_t)((phys ^ (((row >> 1) & 1) << 2)) << 4);
      const uint32_t kl = lds_u + (uint32_t)((stage * KS + k) * KBUF + blk_u * 1024);
      const uint32_t vl = lds_u + (uint32_t)(VREG + (stage * KS + k) * VBUF + blk_u * 1024);
      asm volatile("global_load_lds_dwordx4 %0, %1" : : "v"(kofs), "s"(kbase), "{m0}"(kl) : "memory");
      asm volatile("global_load_lds_dwordx4 %0, %1" : : "v"(vofs), "s"(vbase), "{m0}"(vl) : "memory");
    }
  };

  f32x16 oacc[HT];
#pragma unroll
  for (int t = 0; t < HT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[t][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;       // running max (raw logits), unnormalised sum
  const float c = p.scale_log2;
  // Key tiles [t_begin, t_end) of this split (balanced; empty when the sample
  // has fewer tiles than splits).
  const int ntiles = (nk + kBKV - 1) / kBKV;
  const int t_begin = sp * ntiles / nsp, t_end = (sp + 1) * ntiles / nsp;
  const int last_kv = (t_end - 1) * kBKV;

  // Per-lane constants of the DMA path's fragment reads: the K swizzle of rows
  // 32*kt + r32, and for the transpose read the source row and column within
  // the lane's 16-lane group (rows kb + vi/4, columns db + 4*(vi%4)).
  const int kswz = (r32 >> 1) & 7;
  const int vi = lane & 15;
  const int vrow = vi >> 2, vswz = ((vi >> 3) & 1) << 2, vcol = 4 * (vi & 3) + 16 * ((lane >> 4) & 1);

  // S^T tiles of the tile in buffer buf: rows = keys 32*kt + ..., cols = this
  // wave's 32 queries.
  auto qk = [&](int buf, f32x16 (&sacc)[2]) {
    const char* Ks = lds + buf * (KBUF + VBUF);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const u32x4 kf = DMA ? *reinterpret_cast<const u32x4*>(Ks + (kt * 32 + r32) * KRS + (((2 * s + g) ^ kswz) << 4))
                             : *reinterpret_cast<const u32x4*>(Ks + (kt * 32 + r32) * KRS + s * 32 + g * 16);
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
          // the first instruction of each tile starts from a zero accumulator
          sacc[kt] = Mfma<T>::mma(a, bq, (s == 0 && u == 0) ? f32x16{} : sacc[kt]);
        }
      }
    }
  };

  // Online softmax of tile t's scores and O^T += V^T P^T with V from buffer buf.
  auto softmax_pv = [&](int t, int buf, f32x16 (&sacc)[2]) {
    const int kv0 = t * kBKV;
    const char* Vt = lds + buf * (KBUF + VBUF) + KBUF;

    // Key of element e: kv0 + 32*kt + 8*(e/4) + 4*g + e%4. Mask the ragged tail.
    if (kv0 + kBKV > nk) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kv0 + kt * 32 + 8 * (e >> 2) + 4 * g + (e & 3) >= nk) sacc[kt][e] = -INFINITY;
    }
    // Max over this lane's 32 scores (two independent v_max3 chains).
    const float m0 = max16(sacc[0]), m1 = max16(sacc[1]);
    float mx = max3(m0, m1, m1);
    // Lazy rescale: move the reference max only when some score exceeds it by
    // more than 2^8 (base 2). m_run is the same in lanes l and l ^ 32 (it only
    // changes here, from the query's full max), so each lane tests its own
    // 32 keys and the wave-wide vote covers the query's other 32; the
    // exchange for the full max is needed only in the (rare) branch.
    if (__builtin_amdgcn_ballot_w64((mx - m_run) * c > kRescaleLog2) != 0) {
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int u = 0; u < HT; ++u)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[u][e] *= alpha;
    }
    const float mc = m_run * c;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float pe = __builtin_amdgcn_exp2f(fmaf(sacc[kt][e], c, -mc));
        sacc[kt][e] = pe;
        if constexpr (ES == 4) l_run += pe;
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
          // Row sum of the probabilities as rounded for the PV product (v_dot2 with 1s).
          const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf, pf, 0, 1), ones, l_run, false);
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf, pf, 2, 3), ones, l_run, false);
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf, pf, 4, 5), ones, l_run, false);
          l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf, pf, 6, 7), ones, l_run, false);
        } else {
          pf = sacc[kt][u];
        }
#pragma unroll
        for (int h = 0; h < HT; ++h) {
          typename Mfma<T>::frag vf;
          if constexpr (DMA) {
            // keys kb..kb+3 and kb+8..kb+11 at column h*32 + (lane%32) through two
            // transpose reads of the row-major V tile (K-slot order of P).
            const int kb = kt * 32 + 16 * u + 4 * g, col = h * 32 + vcol;
            const char* a0 = Vt + (kb + vrow) * (HD * ES) + ((((col >> 3) ^ vswz)) << 4) + (col & 7) * ES;
            const auto lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)a0);
            const auto hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(a0 + 8 * HD * ES));
            vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          } else if constexpr (ES == 2) {
            const char* vrow = Vt + (h * 32 + r32) * VRS;
            const int key0 = kt * 32 + 16 * u + 4 * g;
            const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + key0 * ES);
            const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + (key0 + 8) * ES);
            vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
          } else {
            const char* vrow = Vt + (h * 32 + r32) * VRS;
            const int key = kt * 32 + 8 * (u >> 2) + 4 * g + (u & 3);
            vf = *reinterpret_cast<const float*>(vrow + key * ES);
          }
          oacc[h] = Mfma<T>::mma(vf, pf, oacc[h]);
        }
      }
  };
  auto compute = [&](int t, int buf) {
    f32x16 sacc[2];
    qk(buf, sacc);
    softmax_pv(t, buf, sacc);
  };

  if constexpr (DMA) {
    // Five buffers, tile t in buffer (t - t_begin) % 5, loads three tiles
    // ahead. Iteration t waits for tile t + 1 (tile t + 2 stays in flight);
    // its barrier makes every wave's DMA visible and retires the buffer of
    // tile t - 2 (last read by the PV product of iteration t - 1), which
    // receives tile t + 3 (clamped: past the end the last tile is re-read).
    // The matrix cores then take the scores of tile t + 1 and the PV product
    // of tile t - 1 while the vector unit computes the probabilities of tile
    // t: the three are independent, so the steady-state iteration is one
    // basic block the scheduler can interleave. The first and last tiles are
    // peeled. Probabilities use a reference max that moves only in the rare
    // fix-up branch (kTileSumLimit), so no per-tile max is computed.
    const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
    f32x16 minit;                        // -(reference max) * c in every slot
#pragma unroll
    for (int e = 0; e < 16; ++e) minit[e] = 0.0f;
    auto qk2 = [&](int buf, f32x16 (&s)[2]) {
      const char* Ks = lds + (buf * KS + kgrp) * KBUF;
      u32x4 kf[2][NKS];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int q = 0; q < NKS; ++q)
          kf[kt][q] = *reinterpret_cast<const u32x4*>(Ks + (kt * 32 + r32) * KRS + (((2 * q + g) ^ kswz) << 4));
      // All eight reads go out before the first MFMA (left to itself the
      // scheduler pairs each read with its MFMAs, one LDS latency per pair).
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < NKS; ++q)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          s[kt] = Mfma<T>::mma(__builtin_bit_cast(bf16x8, kf[kt][q]), __builtin_bit_cast(bf16x8, qf[q]),
                               q == 0 ? minit : s[kt]);
    };
    // O^T += V^T P^T for the tile in buffer buf; keys kb..kb+3 and kb+8..kb+11
    // at column h*32 + (lane%32) through two transpose reads of the row-major
    // V tile (the K-slot order of P). As for the scores, every fragment read
    // is issued before the first MFMA (2-3% faster at 9831 and 32768 tokens
    // than the scheduler's read-per-MFMA order; same instructions and results).
    auto pv2 = [&](int buf, const bf16x8 (&pf)[2][2]) {
      const char* Vt = lds + VREG + (buf * KS + kgrp) * VBUF;
      bf16x8 vfs[2][2][HT];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int h = 0; h < HT; ++h) {
            const int kb = kt * 32 + 16 * u + 4 * g, col = h * 32 + vcol;
            const char* a0 = Vt + (kb + vrow) * (HD * ES) + (((col >> 3) ^ vswz) << 4) + (col & 7) * ES;
            const auto lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)a0);
            const auto hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(a0 + 8 * HD * ES));
            vfs[kt][u][h] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int h = 0; h < HT; ++h) oacc[h] = Mfma<T>::mma(vfs[kt][u][h], pf[kt][u], oacc[h]);
    };
    // Keys of element e: kv0 + 32*kt + 8*(e/4) + 4*g + e%4; mask those past nk.
    auto mask2 = [&](int t, f32x16 (&s)[2]) {
      const int kv0 = t * kBKV;
      if (kv0 + kBKV > nk) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kv0 + kt * 32 + 8 * (e >> 2) + 4 * g + (e & 3) >= nk) s[kt][e] = -INFINITY;
      }
    };
    // Probabilities 2^((s - m_run) c) as the bf16 P fragments (the shift is
    // already in the accumulators; c is 1 with pre-scaled queries); returns their
    // sum as rounded for the PV product (v_dot2 with ones).
    auto probs = [&](const f32x16 (&s)[2], bf16x8 (&pf)[2][2]) {
      // with key groups a group's only tile can lie past the end (all keys
      // masked, max -inf): its probabilities are then 0
      float part[4];                     // four independent accumulation chains
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            pf[kt][u][e] = (bf16)__builtin_amdgcn_exp2f(QS ? s[kt][8 * u + e] : s[kt][8 * u + e] * c);
          const bf16x8& f = pf[kt][u];
          // the chain's first dot in the three-operand form with a zero
          // accumulator (no register to clear first); the nop covers a dot
          // result read by the next dot as its accumulator
          float a;
          {
            const bf16x2 f01 = __builtin_shufflevector(f, f, 0, 1);
            asm("v_dot2_f32_bf16 %0, %1, %2, 0\n\ts_nop 1" : "=v"(a) : "v"(f01), "v"(ones));
          }
          a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(f, f, 2, 3), ones, a, false);
          a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(f, f, 4, 5), ones, a, false);
          part[2 * kt + u] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(f, f, 6, 7), ones, a, false);
        }
      return (part[0] + part[1]) + (part[2] + part[3]);
    };
    // The query's max over this tile (both key halves of the wave).
    auto tile_max = [&](const f32x16 (&s)[2]) {
      const float m0 = max16(s[0]), m1 = max16(s[1]);
      const float mx = max3(m0, m1, m1);
      return fmaxf(mx, __shfl_xor(mx, 32));
    };
    // Rare: some lane's probabilities outgrew the reference; move it to the
    // tile's max, rescale what was accumulated (including the PV product of
    // the previous tile, issued before) and redo the tile.
    auto fixup = [&](f32x16 (&s)[2], f32x16* next, bf16x8 (&pf)[2][2], float& lt) {
      if (__builtin_amdgcn_ballot_w64(lt > kTileSumLimit) != 0) {
        const float tm = fmaxf(tile_max(s), 0.0f);   // tile max above the reference
        const float alpha = __builtin_amdgcn_exp2f(QS ? -tm : -tm * c);
        m_run += tm;
        l_run *= alpha;
#pragma unroll
        for (int u = 0; u < HT; ++u)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[u][e] *= alpha;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          minit[e] = -m_run;
          s[0][e] -= tm;
          s[1][e] -= tm;
          if (next) {
            next[0][e] -= tm;
            next[1][e] -= tm;
          }
        }
        lt = probs(s, pf);
      }
    };
    auto bnext = [](int b, int k) { b += k; return b >= NBUF ? b - NBUF : b; };
    // Steps i = 0, 1, ...: this wave's tile is t_begin + KS*i + kgrp; stage i
    // % NBUF holds the KS tiles of step i. Loads run DIST steps ahead; a step's
    // barrier retires the stage of step i - 2 (read by the PV product of step
    // i - 1 at the latest), which receives step i + DIST.
    constexpr int DIST = NBUF - 2;
    constexpr int DS = KS * 2 * DQ;                     // DMA instructions per step and wave
    const int n_steps = (t_end - t_begin + KS - 1) / KS;
    auto tile_of = [&](int i) { return t_begin + KS * i + kgrp; };
    auto fetch_step = [&](int i, int stage) {
#pragma unroll
      for (int k = 0; k < KS; ++k) fetch_dma(min((t_begin + KS * i + k) * kBKV, last_kv), stage, k);
    };
    // Step i with S(i) in cur and P(i-1) in pprev: S(i+1) -> next, P(i) -> pcur.
    auto mid = [&](int i, int buf, f32x16 (&cur)[2], f32x16 (&next)[2], const bf16x8 (&pprev)[2][2],
                   bf16x8 (&pcur)[2][2], auto first) {
      wait_vm<(DIST - 2) * DS>();
      __syncthreads();
      fetch_step(i + DIST, bnext(buf, DIST));
      qk2(bnext(buf, 1), next);
      if constexpr (!decltype(first)::value) pv2(bnext(buf, NBUF - 1), pprev);
      float lt = probs(cur, pcur);
      fixup(cur, next, pcur, lt);
      l_run += lt;
    };
    // Last step i (its tiles maybe ragged or past the end): PV(i-1), P(i), then PV(i).
    auto last = [&](int i, int buf, f32x16 (&cur)[2], const bf16x8 (&pprev)[2][2], bf16x8 (&pcur)[2][2],
                    auto first) {
      if constexpr (!decltype(first)::value) pv2(bnext(buf, NBUF - 1), pprev);
      mask2(tile_of(i), cur);
      float lt = probs(cur, pcur);
      fixup(cur, nullptr, pcur, lt);
      l_run += lt;
      pv2(buf, pcur);
    };
    if (t_begin < t_end) {               // uniform over the workgroup
      // Q first: otherwise the compiler, which does not see the DMA, keeps its
      // wait for the Q fragments inside the loop as a full vmcnt(0).
      __builtin_amdgcn_sched_barrier(0);
      wait_vm<0>();
#pragma unroll
      for (int i = 0; i < DIST; ++i) fetch_step(i, i);
      wait_vm<(DIST - 1) * DS>();
      __syncthreads();
      f32x16 sa[2], sb[2];
      bf16x8 pa[2][2], pb[2][2];
      qk2(0, sa);
      if (n_steps == 1) mask2(tile_of(0), sa);
      m_run = tile_max(sa);              // reference max: the first tile's
      {
        const float sub = m_run == -INFINITY ? 0.0f : m_run;   // a key group's tile may lie past the end
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          minit[e] = -sub;
          sa[0][e] -= sub;
          sa[1][e] -= sub;
        }
      }
      const std::true_type yes{};
      const std::false_type no{};
      if (n_steps == 1) {
        last(0, 0, sa, pb, pa, yes);
      } else {
        mid(0, 0, sa, sb, pb, pa, yes);                // S(1) in sb, P(0) in pa
        int i = 1, buf = 1;
        if constexpr (NBUF == 5) {
          // ten steps per round with literal stages: their offsets fold into the reads
          for (; i + 10 < n_steps; i += 10) {
            mid(i, 1, sb, sa, pa, pb, no);
            mid(i + 1, 2, sa, sb, pb, pa, no);
            mid(i + 2, 3, sb, sa, pa, pb, no);
            mid(i + 3, 4, sa, sb, pb, pa, no);
            mid(i + 4, 0, sb, sa, pa, pb, no);
            mid(i + 5, 1, sa, sb, pb, pa, no);
            mid(i + 6, 2, sb, sa, pa, pb, no);
            mid(i + 7, 3, sa, sb, pb, pa, no);
            mid(i + 8, 4, sb, sa, pa, pb, no);
            mid(i + 9, 0, sa, sb, pb, pa, no);
          }
        }
        for (; i + 2 < n_steps; i += 2, buf = bnext(buf, 2)) {
          mid(i, buf, sb, sa, pa, pb, no);
          mid(i + 1, bnext(buf, 1), sa, sb, pb, pa, no);
        }
        if (i + 1 < n_steps) {
          mid(i, buf, sb, sa, pa, pb, no);
          last(i + 1, bnext(buf, 1), sa, pb, pa, no);
        } else {
          last(i, buf, sb, pa, pb, no);
        }
      }
      // no DMA may still target this workgroup's LDS when it retires
      wait_vm<0>();
    }
    if constexpr (KS > 1) {
      // Merge the key groups' (max, sum, output) through LDS, in group order:
      // M = max(m_0, m_1), each group weighted by 2^((m_k - M) c).
      __syncthreads();                   // every wave past its last tile read
      float* xs = reinterpret_cast<float*>(lds) + (size_t)qw * (16 * HT + 2) * 64;
      if (kgrp == 1) {
#pragma unroll
        for (int u = 0; u < HT; ++u)
#pragma unroll
          for (int e = 0; e < 16; ++e) xs[(16 * u + e) * 64 + lane] = oacc[u][e];
        xs[16 * HT * 64 + lane] = m_run;
        xs[(16 * HT + 1) * 64 + lane] = l_run;
      }
      __syncthreads();
      if (kgrp == 1) return;
      const float m1 = xs[16 * HT * 64 + lane], l1 = xs[(16 * HT + 1) * 64 + lane];
      const float mm = fmaxf(m_run, m1);
      const float a0 = __builtin_amdgcn_exp2f((m_run - mm) * c);
      const float a1 = m1 == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((m1 - mm) * c);
#pragma unroll
      for (int u = 0; u < HT; ++u)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[u][e] = oacc[u][e] * a0 + xs[(16 * u + e) * 64 + lane] * a1;
      l_run = l_run * a0 + l1 * a1;
      m_run = mm;
    }
  } else {
    // Fetches are unconditional (past the end they re-read the last tile), so
    // the wait before staging tile t+1 does not cover the loads of tile t+2.
    auto tile = [&](int t, int r) {      // r = (t - t_begin) & 1 (a constant at each call site)
      fetch(min(t * kBKV + 2 * kBKV, last_kv), r);
      compute(t, r);
      stage(r ^ 1, r ^ 1);
      __syncthreads();
    };
    if (t_begin < t_end) {               // uniform over the workgroup
      fetch(t_begin * kBKV, 0);
      fetch(min((t_begin + 1) * kBKV, last_kv), 1);
      stage(0, 0);
      __syncthreads();
      int t = t_begin;
      for (; t + 1 < t_end; t += 2) {
        tile(t, 0);
        tile(t + 1, 1);
      }
      if (t < t_end) tile(t, 0);
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!q_ok) return;
  if constexpr (SPLIT) {
    const size_t prow = ((size_t)sp * p.rows + (q_begin - p.qs.off[0] + qi)) * p.heads + head;
    float* po = p.part_o + prow * HD;
#pragma unroll
    for (int h = 0; h < HT; ++h)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<float4*>(po + h * 32 + 8 * q4 + 4 * g) =
            make_float4(oacc[h][4 * q4], oacc[h][4 * q4 + 1], oacc[h][4 * q4 + 2], oacc[h][4 * q4 + 3]);
    if (g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m_run * c, l_tot);
    return;
  }
  const float inv = 1.0f / l_tot;
  T* orow = reinterpret_cast<T*>(p.o + ((size_t)(q_begin + qi) * p.ldo + head * HD) * ES);
#pragma unroll
  for (int h = 0; h < HT; ++h)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = oacc[h][4 * q4 + e] * inv;
      T* dst = orow + h * 32 + 8 * q4 + 4 * g;
      if constexpr (ES == 2) {
        bf16x4 o4;
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (bf16)v[e];
        *reinterpret_cast<bf16x4*>(dst) = o4;
      } else {
        *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
}

// Merge of the key-range splits: one thread per (query row, head, 4 output
// columns). With M = max_s m_s, w_s = 2^(m_s - M): o = sum_s w_s O_s / sum_s w_s l_s.
template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs p) {
  constexpr int D4 = HD / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)p.rows * p.heads * D4) return;
  const int d = (int)(i % D4) * 4;
  const int64_t rh = i / D4;                           // row * heads + head
  const int head = (int)(rh % p.heads);
  const int64_t row = rh / p.heads;
  const size_t split_stride = (size_t)p.rows * p.heads;
  float mx = -INFINITY;
  for (int s = 0; s < p.splits; ++s) mx = fmaxf(mx, p.part_ml[(s * split_stride + rh) * 2]);
  float l = 0.0f;
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int s = 0; s < p.splits; ++s) {
    const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + (s * split_stride + rh) * 2);
    const float w = exp2f(ml.x - mx);                  // 0 for an empty split (max -inf)
    const float4 o = *reinterpret_cast<const float4*>(p.part_o + (s * split_stride + rh) * HD + d);
    l += w * ml.y;
    acc.x += w * o.x;
    acc.y += w * o.y;
    acc.z += w * o.z;
    acc.w += w * o.w;
  }
  const float inv = 1.0f / l;
  T* dst = reinterpret_cast<T*>(p.o) + (size_t)(p.qs.off[0] + row) * p.ldo + head * HD + d;
  if constexpr (sizeof(T) == 2) {
    bf16x4 o4;
    o4[0] = (bf16)(acc.x * inv);
    o4[1] = (bf16)(acc.y * inv);
    o4[2] = (bf16)(acc.z * inv);
    o4[3] = (bf16)(acc.w * inv);
    *reinterpret_cast<bf16x4*>(dst) = o4;
  } else {
    *reinterpret_cast<float4*>(dst) = make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  }
}

template <typename T, int HD, int NW, int SITE, int KS = 1, bool QS = false>
hipError_t launch_k(const AttnArgs& a, int tiles, hipStream_t s) {
  const dim3 block(64 * NW);
  if constexpr (KS > 1) {
    if (a.splits != 1) return hipErrorInvalidValue;
    launch((k_attn<T, HD, NW, SITE, false, KS, QS>), dim3(tiles * a.heads), block, 0, s, a);
    return hipGetLastError();
  }
  if (a.splits == 1) {
    launch((k_attn<T, HD, NW, SITE, false, 1, QS>), dim3(tiles * a.heads), block, 0, s, a);
    return hipGetLastError();
  }
  launch((k_attn<T, HD, NW, SITE, true, 1, QS>), dim3(tiles * a.heads * a.splits), block, 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)a.rows * a.heads * (HD / 4);
  launch((k_attn_combine<T, HD>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// splits > 1 requires a.part_o / a.part_ml sized for them.
template <int NW, int SITE, int KS = 1>
hipError_t launch_a(int dt, int hd, const AttnArgs& a0, int heads, int splits, hipStream_t s, bool qs) {
  AttnArgs a = a0;
  constexpr int BQ = 32 * NW / KS;
  a.tile_off[0] = 0;
  for (int b = 0; b < a.qs.B; ++b) a.tile_off[b + 1] = a.tile_off[b] + (a.qs.off[b + 1] - a.qs.off[b] + BQ - 1) / BQ;
  const int tiles = a.tile_off[a.qs.B];
  if (tiles == 0) return hipSuccess;
  a.heads = heads;
  a.splits = splits;
  a.rows = a.qs.off[a.qs.B] - a.qs.off[0];
  if constexpr (KS > 1) {
    if (dt == DT_BF16 && hd == 64)
      return qs ? launch_k<bf16, 64, NW, SITE, KS, true>(a, tiles, s) : launch_k<bf16, 64, NW, SITE, KS>(a, tiles, s);
    return hipErrorInvalidValue;
  } else {
    if (dt == DT_BF16 && hd == 64)
      return qs ? launch_k<bf16, 64, NW, SITE, 1, true>(a, tiles, s) : launch_k<bf16, 64, NW, SITE>(a, tiles, s);
    if (dt == DT_BF16 && hd == 32) return launch_k<bf16, 32, NW, SITE>(a, tiles, s);
    if (dt == DT_F32 && hd == 64) return launch_k<float, 64, NW, SITE>(a, tiles, s);
    if (dt == DT_F32 && hd == 32) return launch_k<float, 32, NW, SITE>(a, tiles, s);
    return hipErrorInvalidValue;
  }
}

// Bytes of split partials for `splits` splits of `rows` query rows.
inline size_t split_bytes(int splits, int rows, int heads, int hd) {
  return (size_t)splits * rows * heads * (hd + 2) * sizeof(float);
}

// 8 waves (256 queries) per workgroup when that still gives at least 160
// workgroups; measured on MI355X from 300 to 4096 queries, 256-query
// workgroups lead from about 2300 queries up (eight waves share each staged
// K/V tile, which halves the staging work per query). Below that the time is
// the serial chain of key tiles that one wave walks. Two ways shorten it:
//  * key groups (bf16, 64-wide heads): the waves of a workgroup split into two
//    key groups merged through LDS; 64-query workgroups of four waves while
//    they fit one round on the 256 CUs (128 KiB of LDS: one per CU), else
//    128-query workgroups of eight waves. Chain: half the key tiles.
//  * key-range splits over workgroups of four waves, merged by a second
//    kernel, while all of them fit one round and every split keeps at least
//    8 key tiles. Chain: 1/splits of the key tiles, plus the merge.
// Measured on MI355X, 16 heads: both cost about 0.85 us per tile of chain,
// and splits about 4.5 us more in fixed cost, so key groups are taken unless
// splits shorten the chain by more than kSplitGainTiles. Examples: self 820
// queries 10.7 us (key groups) against 13.6 (eight waves, key groups); cross
// 820 x 1374 keys 14.6 against 19.2 (two splits); 64 x 4096 keys 29.7 against
// 16.4 (eight splits). Other types and head sizes: four waves, with splits.
constexpr long kSplitGainTiles = 5;

template <int SITE>
hipError_t launch_site(int dt, int hd, const AttnArgs& a, int heads, float* ws, size_t ws_bytes, hipStream_t s,
                       bool qs) {
  long t64 = 0, t128 = 0, t256 = 0, kt_min = 1L << 30, kt_max = 0;
  for (int b = 0; b < a.qs.B; ++b) {
    const int nq = a.qs.off[b + 1] - a.qs.off[b];
    if (nq == 0) continue;
    t64 += (nq + 63) / 64;
    t128 += (nq + 127) / 128;
    t256 += (nq + 255) / 256;
    const long kt = (a.ks.off[b + 1] - a.ks.off[b] + kBKV - 1) / kBKV;
    kt_min = std::min(kt_min, kt);
    kt_max = std::max(kt_max, kt);
  }
  // The DMA path addresses a sample's key and value rows with 32-bit offsets
  // from the sample's first row.
  if (dt == DT_BF16 && hd == 64 && kt_max * kBKV * (int64_t)std::max(a.ldk, a.ldv) * 2 >= (int64_t(1) << 31))
    return hipErrorInvalidValue;
  if (t256 * heads >= 160) return launch_a<8, SITE>(dt, hd, a, heads, 1, s, qs);
  int splits = 1;
  while (splits < 8 && t128 * heads * splits * 2 <= 256 && kt_min >= 16 * splits) splits *= 2;
  const int rows = a.qs.off[a.qs.B] - a.qs.off[0];
  while (splits > 1 && (!ws || split_bytes(splits, rows, heads, hd) > ws_bytes)) splits /= 2;
  if (dt == DT_BF16 && hd == 64 && (kt_max + 1) / 2 - (kt_max + splits - 1) / splits <= kSplitGainTiles) {
    if (t64 * heads <= 256) return launch_a<4, SITE, 2>(dt, hd, a, heads, 1, s, qs);
    return launch_a<8, SITE, 2>(dt, hd, a, heads, 1, s, qs);
  }
  AttnArgs b = a;
  if (splits > 1) {
    b.part_o = ws;
    b.part_ml = ws + (size_t)splits * rows * heads * hd;
  }
  return launch_a<4, SITE>(dt, hd, b, heads, splits, s, qs);
}

}  // namespace

hipError_t launch_attention(int site, int dt, int heads, int hd, const Segs& qs, const Segs& ks, const void* q,
                            int ldq, const void* k, int ldk, const void* v, int ldv, void* o, int ldo, float* ws,
                            size_t ws_bytes, hipStream_t s, bool q_scaled) {
  AttnArgs a;
  a.qs = qs;
  a.ks = ks;
  a.q = (const char*)q;
  a.k = (const char*)k;
  a.v = (const char*)v;
  a.o = (char*)o;
  a.ldq = ldq;
  a.ldk = ldk;
  a.ldv = ldv;
  a.ldo = ldo;
  a.scale_log2 = q_scaled ? 1.0f : attention_q_scale(hd);
  a.splits = 1;
  a.part_o = a.part_ml = nullptr;
  if (site == SITE_SELF) return launch_site<SITE_SELF>(dt, hd, a, heads, ws, ws_bytes, s, q_scaled);
  if (site == SITE_CROSS) return launch_site<SITE_CROSS>(dt, hd, a, heads, ws, ws_bytes, s, q_scaled);
  return launch_site<SITE_OP>(dt, hd, a, heads, ws, ws_bytes, s, q_scaled);
}

}  // namespace f3c
