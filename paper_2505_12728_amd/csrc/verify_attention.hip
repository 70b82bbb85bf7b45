// Verification attention of the drafted block over the KV cache (SpecFLASH
// Sec. 3.1: the target scores all K drafted tokens in one parallel pass).
//
// The work is HBM-bound: every key / value of the cache is read once for
// all k * g query rows that share a KV head (k block positions times g
// grouped query heads), so the design keeps those rows resident and streams
// the cache.
//
// Kernel 1 (split): grid (split, KV head x row group, sequence), 4 waves.
//   Each work-group owns one contiguous key range of one (sequence, KV head)
//   and up to 64 query rows; its 4 waves take interleaved 32-key tiles.
//   Per tile a wave
//     - loads K as matrix-core A fragments straight from HBM (16 bytes per
//       lane, 8 contiguous channels of one key), and V in coalesced 16-byte
//       pieces that it stages in its own LDS slice;
//     - computes S^T = K Q^T on bf16 matrix cores, so that every lane holds
//       scores of exactly one query row (column c of the accumulator);
//     - runs the online softmax in fp32 (base-2 exponent, masked by the
//       causal limit kv_len - k + j of its row);
//     - accumulates O^T += V^T P^T, reading V^T fragments from LDS with the
//       transposing ds_read_tr16_b64, and feeding P as a bf16 hi + lo pair
//       (P = hi + lo to ~2^-16 relative), which keeps the result within the
//       float tolerance of the fp32 reference without converting V.
//   The 4 waves then merge their (max, sum, O) through LDS in a fixed order
//   and write one normalised partial (o, lse) per split.
// Kernel 2 (merge): combines the splits of each row with the log-sum-exp
//   rule and writes out / lse in the caller's [B, k, Hq] layout.
//
// fp32 caches take a plain (non matrix-core) split kernel with the same
// partial format; it computes in float64 so fp32 inputs keep fp32 accuracy.
#include <math.h>

#include <algorithm>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

constexpr int kTile = 32;       // keys per tile of the bf16 kernel

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;

// Offset (in elements) of the D-channel slice of token t, KV head hk.
template <bool PAGED>
__device__ __forceinline__ size_t kv_offset(const VerifyArgs& a, int b, int hk, int t, int D) {
  if constexpr (PAGED) {
    int page = a.page_table[(size_t)b * a.max_pages + (t >> 4)];
    page = min(max(page, 0), a.num_pages - 1);
    return (((size_t)page * a.Hkv + hk) * 16 + (t & 15)) * (size_t)D;
  } else {
    return (((size_t)b * a.Lmax + t) * a.Hkv + hk) * (size_t)D;
  }
}

__device__ __forceinline__ int seq_len(const VerifyArgs& a, int b, bool paged) {
  const int cap = paged ? a.max_pages * 16 : a.Lmax;
  return min(max(a.kv_len[b], 0), cap);
}

// ----------------------------------------------------------- bf16 split
// One work-group = NW waves = NW 16-row blocks of one (sequence, KV head,
// key split).  All waves walk the same 32-key tiles.  Tiles are copied
// HBM -> LDS by the global_load_lds DMA (no VGPR staging) into a ring of
// NBUF buffers, NBUF - 1 tiles ahead of the compute; with two or three
// work-groups per compute unit about 96 KB per unit is in flight.  Each key
// row keeps its 16-byte pieces XOR-swizzled by lds_swizzle(key), so the
// K-fragment reads (16 keys x one piece) and the transposed V reads (4 keys
// x 8 bytes per 16 lanes) are free of bank conflicts.
//
// Per tile a wave does 8 + 16 matrix-core ops and little else: the causal
// mask is applied only on the tail tile, the running maximum is raised (and
// O, l rescaled) only when a row's scores exceed it by more than 2^8 (the
// stale maximum is exact for the final o = O / l; p stays below 256), and
// copy addresses are per-lane constants plus a per-tile scalar offset.
template <int D, int NW, bool PAGED, int KG>
__global__ __launch_bounds__(NW * 64) void verify_split_bf16(VerifyArgs a, int keys_per_split,
                                                             int nsplit, int row_groups,
                                                             int rows_padded) {
  constexpr int TK = kTile;
  constexpr int DC = D / 32;                   // 32-channel K slices (QK^T)
  constexpr int DB = D / 16;                   // 16-channel output blocks (PV)
  constexpr int PK = D / 8;                    // 16-byte pieces per key row
  constexpr int ROW_BYTES = D * 2;
  constexpr int HALF_BYTES = TK * ROW_BYTES;   // K (or V) part of a buffer
  constexpr int BUF_BYTES = 2 * HALF_BYTES;
  constexpr int DMA_PER_HALF = TK * PK / 64;   // 64-lane copies per K (or V) tile
  constexpr int DMA_PER_WAVE = 2 * DMA_PER_HALF / NW;   // per tile
  constexpr int NWR = NW / KG;                 // waves per key group = 16-row blocks
  static_assert((2 * DMA_PER_HALF) % NW == 0, "tile copy must split evenly");
  static_assert(NW % KG == 0 && (KG == 1 || KG == 2), "key groups");
  static_assert(TK == 32, "one P V step per tile");
  // ring depth: NBUF - KG tiles in flight.  KG = 1: two (NW = 4) or three
  // (NW < 4) work-groups share a compute unit, so every SIMD runs two or
  // more waves.  KG = 2: one work-group of 8 waves per unit, the two groups
  // of 4 waves taking alternate tiles of one deep ring (one long key stream
  // per unit, two waves per SIMD).
  constexpr int NBUF = KG == 2 ? 8 : ((NW == 4) ? 4 : 3);
  static_assert(NBUF % KG == 0 && (NBUF - 2 * KG) * DMA_PER_WAVE < 64, "vmcnt range");
  constexpr float kRescale = 8.f;              // log2 headroom before rescaling
  __shared__ __align__(16) unsigned char ring[NBUF][BUF_BYTES];

  // grid (KV head x row group, split, sequence): the work-groups of one key
  // range are dispatched together, so the heads of a key read their
  // interleaved cache rows at about the same time
  const int split = blockIdx.y;
  const int hk = blockIdx.x / row_groups;
  const int rg = blockIdx.x % row_groups;
  const int b = blockIdx.z;
  const int L = seq_len(a, b, PAGED);
  const int k0 = split * keys_per_split;
  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, G = lane >> 4, c = lane & 15;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int wr = w % NWR, kgrp = w / NWR;      // row block, key group
  const int rblk = rg * NWR * 16 + wr * 16;    // this wave's first row
  if (k0 >= L) {
    // empty split: the merge skips it; with a single split (nothing to
    // merge) this work-group writes its rows directly: o = 0, lse = -inf
    if (nsplit == 1 && split == 0 && kgrp == 0 && rblk + c < R) {
      const int r = rblk + c;
      const int j = r / g;
      const int orow = (b * a.k + j) * a.Hq + hk * g + (r - j * g);
      for (int d4 = G; d4 < D / 4; d4 += 4)
        *reinterpret_cast<floatx4*>(a.out + (size_t)orow * D + d4 * 4) = floatx4{0.f, 0.f, 0.f, 0.f};
      if (a.lse != nullptr && G == 0) a.lse[orow] = -INFINITY;
    }
    return;
  }
  const int k1 = min(L, k0 + keys_per_split);
  // a wave whose rows are all padding (R not a multiple of 16 * NWR) runs
  // the same loop on zero queries and writes nothing
  const bool active = rblk < R;                // wave-uniform

  // This lane's query row r = rblk + c: block position j = r / g, query head
  // hk * g + r % g.  B operand of S^T = K Q^T.
  bf16x8 qf[DC];
  int lim = -1;
  int orow = -1;
  {
    const int r = rblk + c;
    Pack8 pk;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      pk.u = u32x4{0u, 0u, 0u, 0u};
      qf[dc] = pk.b;
    }
    if (r < R) {
      const int j = r / g;
      const int h = hk * g + (r - j * g);
      orow = (b * a.k + j) * a.Hq + h;
      const u32x4* src = reinterpret_cast<const u32x4*>(
          static_cast<const uint16_t*>(a.q) + (size_t)orow * D);
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        pk.u = src[dc * 4 + G];
        qf[dc] = pk.b;
      }
      lim = L - a.k + j;                       // last visible key of this row
    }
  }
  // every row sees keys 0 .. L - k; tiles ending there need no mask
  const int unmasked_end = L - a.k;

  float m = -INFINITY, l = 0.f;
  floatx4 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = floatx4{0.f, 0.f, 0.f, 0.f};

  const uint16_t* kbase = static_cast<const uint16_t*>(a.kc);
  const uint16_t* vbase = static_cast<const uint16_t*>(a.vc);
  const int ntiles = (k1 - k0 + TK - 1) / TK;
  const int last = ntiles - 1;

  // Copy i of this wave (ii = w * DMA_PER_WAVE + i) covers half
  // ii / DMA_PER_HALF (K or V) and pieces P = (ii % DMA_PER_HALF) * 64 +
  // lane: key P / PK, LDS slot P % PK holding global piece slot ^ lds_swizzle(key).
  // Its source is a per-lane constant plus a per-tile offset, except in the
  // tail tile, where keys past the sequence re-read its last key (masked).
  // Page ids are scalar loads, so they do not count against vmcnt.
  size_t cbase[DMA_PER_WAVE];
  int ckey[DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < DMA_PER_WAVE; ++i) {
    const int ii = w * DMA_PER_WAVE + i;
    const int P = (ii % DMA_PER_HALF) * 64 + lane;
    const int key = P / PK, piece = P % PK;
    ckey[i] = key;
    const size_t pieceoff = (size_t)((piece ^ lds_swizzle<PK>(key)) * 8);
    if constexpr (PAGED)
      cbase[i] = (((size_t)hk * 16 + (key & 15)) * D) + pieceoff;
    else
      cbase[i] = (((size_t)b * a.Lmax + k0 + key) * a.Hkv + hk) * (size_t)D + pieceoff;
  }
  const size_t tile_stride = (size_t)TK * a.Hkv * D;   // contiguous: elements per tile
  auto issue = [&](int tile, unsigned char* slot) {
    const int t0 = k0 + tile * TK;
    const bool tail = t0 + TK > L;
    int pg0 = 0, pg1 = 0;
    if constexpr (PAGED) {
      // the page table is read-only here: constant-space loads become
      // scalar loads, which leave the vector-memory counter to the copies
      const __attribute__((address_space(4))) int32_t* pt =
          (const __attribute__((address_space(4))) int32_t*)(a.page_table + (size_t)b * a.max_pages);
      const int lastp = (L - 1) >> 4;
      pg0 = min(max((int)pt[min(t0 >> 4, lastp)], 0), a.num_pages - 1);
      pg1 = min(max((int)pt[min((t0 >> 4) + 1, lastp)], 0), a.num_pages - 1);
    }
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const int ii = w * DMA_PER_WAVE + i;
      const int half = ii / DMA_PER_HALF;
      size_t off;
      if constexpr (PAGED) {
        int key = ckey[i];
        size_t base = cbase[i];
        if (tail && t0 + key > L - 1) {        // re-read the last key
          const int t = L - 1;
          key = t - t0;
          base = (((size_t)hk * 16 + (t & 15)) * D) + (cbase[i] & (size_t)(PK * 8 - 1));
        }
        const int pg = key < 16 ? pg0 : pg1;
        off = base + (size_t)pg * a.Hkv * 16 * D;
      } else {
        off = cbase[i] + (size_t)tile * tile_stride;
        if (tail && t0 + ckey[i] > L - 1)      // re-read the last key
          off -= (size_t)(t0 + ckey[i] - (L - 1)) * a.Hkv * D;
      }
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)((half ? vbase : kbase) + off),
                                       (lds_void*)(slot + half * HALF_BYTES + (ii % DMA_PER_HALF) * 1024),
                                       16, 0, 0);
    }
  };

  // per-lane LDS offsets of the fragment reads inside a buffer
  uint32_t koff[2][DC];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      const int key = kb * 16 + c;
      koff[kb][dc] = key * ROW_BYTES + (((dc * 4 + G) ^ lds_swizzle<PK>(key)) * 16);
    }
  // ds_read_tr16_b64: lane j of group G addresses key 4G + j/4 (+16) at
  // channels db*16 + 4*(j%4); lane c then receives 4 keys at channel db*16 + c
  uint32_t voff[2][DB];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int key = hh * 16 + 4 * G + (c >> 2);
      const int ch = db * 16 + 4 * (c & 3);
      voff[hh][db] = HALF_BYTES + key * ROW_BYTES + (((ch >> 3) ^ lds_swizzle<PK>(key)) * 16) + (ch & 7) * 2;
    }

  auto compute = [&](int it, const unsigned char* slot) {
    const uint32_t sb = lds_addr(slot);
    const int t0 = k0 + it * TK;

    u32x4 kr[2][DC];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) kr[kb][dc] = lds_read_b128(sb + koff[kb][dc]);
    lds_wait();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) tie(kr[kb][dc]);
    // V^T fragments for P V, issued now so they overlap the scores
    u32x2 vr[2][DB];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int db = 0; db < DB; ++db) vr[hh][db] = lds_read_tr16_b64(sb + voff[hh][db]);

    // S^T = K Q^T: lane holds S[row c][key t0 + kb*16 + 4G + i] (log2 units)
    float x[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = kr[kb][dc];
        acc = mfma_bf16(pk.b, qf[dc], acc);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) x[kb * 4 + i] = acc[i] * a.scale_log2;
    }
    if (t0 + TK - 1 > unmasked_end) {          // tail tile: causal mask
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int t = t0 + (e >> 2) * 16 + 4 * G + (e & 3);
        if (t > lim) x[e] = -INFINITY;
      }
    }

    // online softmax with a lazily raised maximum
    float tmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                       fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    tmax = wave_max_across_groups(tmax);
    if (__ballot(tmax > m + kRescale) != 0ull) {
      const float mnew = fmaxf(m, tmax);
      const float alpha = (mnew == -INFINITY) ? 1.f : fast_exp2(m - mnew);
      l *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
      m = mnew;
    }
    bf16x8 ph, pl;
    float psum = 0.f;
    const bool none = m == -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pv = none ? 0.f : fast_exp2(x[e] - m);
      psum += pv;
      const __bf16 hi = float_to_bf16(pv);
      ph[e] = hi;
      pl[e] = float_to_bf16(pv - bf16_to_float(hi));
    }
    l += psum;

    // O^T += V^T P^T.  The product's K index runs over keys {4G..4G+3,
    // 16+4G..16+4G+3}, the order in which the score accumulator handed this
    // lane its P values; accumulator element i of block db is channel
    // db*16 + 4G + i of row c.
    lds_wait();
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int db = 0; db < DB; ++db) tie(vr[hh][db]);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      Pack8 vv;
      vv.u = u32x4{vr[0][db][0], vr[0][db][1], vr[1][db][0], vr[1][db][1]};
      o[db] = mfma_bf16(vv.b, ph, o[db]);
      o[db] = mfma_bf16(vv.b, pl, o[db]);
    }
  };

  // Every step issues KG tiles (past the end it re-reads the last one, which
  // is still cached), so exactly (NBUF - 2 KG) tiles' copies are newer than
  // the step's own tiles at each wait, and the wait covers precisely the
  // tiles about to be read; the barrier also frees the slots of the
  // previous step for refilling.  The tile reads are asm, so the compiler
  // adds no waits of its own between them and the copies.
  const int nsteps = (ntiles + KG - 1) / KG;
#pragma unroll
  for (int i = 0; i < NBUF - KG; ++i) issue(min(i, last), ring[i]);
  for (int it = 0; it < nsteps; ++it) {
    wait_vm_then_barrier<(NBUF - 2 * KG) * DMA_PER_WAVE>();
#pragma unroll
    for (int j = 0; j < KG; ++j) {
      const int t = KG * it + NBUF - KG + j;
      issue(min(t, last), ring[t % NBUF]);
    }
    const int mine = KG * it + kgrp;           // wave-uniform
    if (KG == 1 || mine < ntiles) compute(mine, ring[mine % NBUF]);
  }
  // no copy may still be writing this work-group's LDS when it exits
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
  l = wave_sum_across_groups(l);
  if constexpr (KG == 2) {
    // group 1 hands (m, l, O) of its row block to group 0 through the ring
    __syncthreads();                           // every wave is done with the ring
    floatx4* xo = reinterpret_cast<floatx4*>(&ring[0][0]);
    float2* xml = reinterpret_cast<float2*>(&ring[0][0] + NWR * DB * 64 * 16);
    if (kgrp == 1) {
#pragma unroll
      for (int db = 0; db < DB; ++db) xo[(wr * DB + db) * 64 + lane] = o[db];
      xml[wr * 64 + lane] = make_float2(m, l);
    }
    __syncthreads();
    if (kgrp == 1) return;
    const float2 ml = xml[wr * 64 + lane];
    const float mn = fmaxf(m, ml.x);
    const float f0 = m == -INFINITY ? 0.f : fast_exp2(m - mn);
    const float f1 = ml.x == -INFINITY ? 0.f : fast_exp2(ml.x - mn);
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = o[db] * f0 + xo[(wr * DB + db) * 64 + lane] * f1;
    l = l * f0 + ml.y * f1;
    m = mn;
  }
  if (!active) return;

  const float inv = l > 0.f ? 1.f / l : 0.f;
  auto store_row = [&](float* dst) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<floatx4*>(dst + db * 16 + 4 * G) = o[db] * inv;
  };
  if (nsplit == 1) {
    if (orow >= 0) {
      store_row(a.out + (size_t)orow * D);
      if (a.lse != nullptr && G == 0)
        a.lse[orow] = l > 0.f ? (m + log2f(l)) * kLn2 : -INFINITY;
    }
    return;
  }
  const size_t prow = ((size_t)(b * a.Hkv + hk) * nsplit + split) * rows_padded + rblk + c;
  store_row(a.part_o + prow * D);
  if (G == 0) a.part_lse[prow] = l > 0.f ? m + log2f(l) : -INFINITY;
}

// ----------------------------------------------------------- fp32 split
// fp32 inputs: scores, softmax and P V run in float64, so the result keeps
// full fp32 accuracy even when large scores make the softmax sensitive to
// rounding.  Queries and the split's scores sit in LDS; one wave per row
// forms the softmax statistics; threads over (row, channel) accumulate P V.
template <bool PAGED>
__global__ __launch_bounds__(256) void verify_split_f32(VerifyArgs a, int keys_per_split,
                                                        int nsplit, int rows_padded) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int D = a.D;
  const int split = blockIdx.x;
  const int hk = blockIdx.y;
  const int b = blockIdx.z;
  const int L = seq_len(a, b, PAGED);
  const int k0 = split * keys_per_split;
  if (k0 >= L) return;
  const int nk = min(L, k0 + keys_per_split) - k0;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int tid = threadIdx.x;

  double* ss = reinterpret_cast<double*>(smem);        // [R][keys_per_split]
  double* st = ss + (size_t)R * keys_per_split;         // [R][2]: max, sum
  float* qs = reinterpret_cast<float*>(st + 2 * R);     // [R][D]
  const float* qg = static_cast<const float*>(a.q);
  for (int i = tid; i < R * D; i += blockDim.x) {
    const int r = i / D, e = i % D;
    const int j = r / g, h = hk * g + (r - j * g);
    qs[i] = qg[(((size_t)b * a.k + j) * a.Hq + h) * D + e];
  }
  __syncthreads();
  const float* kg = static_cast<const float*>(a.kc);
  const float* vg = static_cast<const float*>(a.vc);
  const double scale = (double)a.scale;
  for (int i = tid; i < nk * R; i += blockDim.x) {
    const int tt = i / R, r = i % R;
    const int t = k0 + tt;
    const int j = r / g;
    double s = -INFINITY;
    if (t <= L - a.k + j) {
      const float* kr = kg + kv_offset<PAGED>(a, b, hk, t, D);
      const float* qr = qs + r * D;
      double acc = 0.0;
      for (int e = 0; e < D; ++e) acc = fma((double)qr[e], (double)kr[e], acc);
      s = acc * scale;
    }
    ss[(size_t)r * keys_per_split + tt] = s;
  }
  __syncthreads();
  const int w = tid >> 6, lane = tid & 63;
  for (int r = w; r < R; r += blockDim.x / kWave) {
    double mx = -INFINITY;
    for (int tt = lane; tt < nk; tt += kWave) mx = fmax(mx, ss[(size_t)r * keys_per_split + tt]);
    for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, 64));
    double sum = 0.0;
    for (int tt = lane; tt < nk; tt += kWave) {
      const double v = ss[(size_t)r * keys_per_split + tt];
      const double p = (mx == -INFINITY) ? 0.0 : exp(v - mx);
      ss[(size_t)r * keys_per_split + tt] = p;
      sum += p;
    }
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
    if (lane == 0) {
      st[2 * r] = mx;
      st[2 * r + 1] = sum;
    }
  }
  __syncthreads();
  const size_t base = ((size_t)(b * a.Hkv + hk) * nsplit + split) * rows_padded;
  for (int i = tid; i < R * D; i += blockDim.x) {
    const int r = i / D, e = i % D;
    const double sum = st[2 * r + 1];
    double acc = 0.0;
    for (int tt = 0; tt < nk; ++tt) {
      const double p = ss[(size_t)r * keys_per_split + tt];
      if (p != 0.0) acc = fma(p, (double)vg[kv_offset<PAGED>(a, b, hk, k0 + tt, D) + e], acc);
    }
    a.part_o[(base + r) * D + e] = sum > 0.0 ? (float)(acc / sum) : 0.f;
    if (e == 0)
      a.part_lse[base + r] =
          sum > 0.0 ? (float)((st[2 * r] + log(sum)) * 1.4426950408889634) : -INFINITY;
  }
}

// ---------------------------------------------------------------- merge
// One wave per output row of one (sequence, KV head).  The lanes load the
// split lse values 64 at a time and form their weights 2^(lse - max) in
// parallel; then the two half-waves take alternate splits (in lockstep, the
// weight of split j handed over by a lane shuffle), each lane
// accumulating 4 channels of the weighted partial outputs (loads of
// several splits in flight), and the halves are added at the end.
// Grid (rows / 4, sequence x KV head).
__global__ __launch_bounds__(256) void verify_merge(VerifyArgs a, int keys_per_split,
                                                    int nsplit, int rows_padded, int paged) {
  const int pair = blockIdx.y;
  const int hk = pair % a.Hkv;
  const int b = pair / a.Hkv;
  const int D = a.D;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + w;
  if (r >= R) return;
  const int L = seq_len(a, b, paged != 0);
  const int nvalid = min(nsplit, (L + keys_per_split - 1) / keys_per_split);
  const size_t base = (size_t)pair * nsplit * rows_padded + r;
  float mx = -INFINITY;
  for (int s = lane; s < nvalid; s += 64) mx = fmaxf(mx, a.part_lse[base + (size_t)s * rows_padded]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  const int half = lane >> 5, d4 = lane & 31;
  const bool active = d4 < D / 4;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  if (mx != -INFINITY) {
    for (int s0 = 0; s0 < nvalid; s0 += 64) {
      const int n = min(64, nvalid - s0);
      float wl = 0.f;
      if (lane < n) {
        const float ls = a.part_lse[base + (size_t)(s0 + lane) * rows_padded];
        wl = ls == -INFINITY ? 0.f : exp2f(ls - mx);
      }
      wsum += wl;
      // both halves run the same trip count, so every shuffle reads an
      // active lane; lanes past the last split (j = n, odd n) get weight 0
      for (int jj = 0; jj < n; jj += 2) {
        const int j = jj + half;
        const float wgt = __shfl(wl, j & 63, 64);
        const size_t pr = base + (size_t)(s0 + j) * rows_padded;
        if (j < n && active && wgt != 0.f)
          acc += wgt * *reinterpret_cast<const floatx4*>(a.part_o + pr * D + d4 * 4);
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) wsum += __shfl_xor(wsum, off, 64);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += __shfl_xor(acc[e], 32, 64);
  }
  const int j = r / g;
  const int h = hk * g + (r - j * g);
  const size_t orow = ((size_t)b * a.k + j) * a.Hq + h;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  if (half == 0 && active) *reinterpret_cast<floatx4*>(a.out + orow * D + d4 * 4) = acc * inv;
  if (a.lse != nullptr && lane == 0)
    a.lse[orow] = wsum > 0.f ? (mx + log2f(wsum)) * kLn2 : -INFINITY;
}

template <int D, int NW, bool PAGED, int KG>
hipError_t launch_bf16(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  dim3 grid(a.Hkv * p.row_groups, p.nsplit, a.B);
  hipLaunchKernelGGL((verify_split_bf16<D, NW, PAGED, KG>), grid, dim3(NW * 64), 0, st, a,
                     p.keys_per_split, p.nsplit, p.row_groups, p.rows_padded);
  return hipGetLastError();
}

template <int D, bool PAGED>
hipError_t dispatch_rb(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  switch (p.row_blocks) {
    case 1: return launch_bf16<D, 1, PAGED, 1>(a, p, st);
    case 2: return launch_bf16<D, 2, PAGED, 1>(a, p, st);
    default: return launch_bf16<D, 8, PAGED, 2>(a, p, st);
  }
}

}  // namespace

VerifyPlan plan_verify(int B, int k, int Hq, int Hkv, int D, int capacity, int dtype) {
  VerifyPlan p{};
  p.g = Hq / Hkv;
  p.rows = k * p.g;
  p.capacity = capacity;
  const int blocks16 = (p.rows + 15) / 16;
  if (dtype == 0) {  // fp32 path: all rows in one work-group
    p.row_blocks = blocks16;
    p.row_groups = 1;
    p.rows_padded = p.rows;
    // fp32 queries, fp64 scores of all rows for one split and fp64 row
    // statistics stay within 64 KB of LDS
    int kps = ((65536 - 4 * p.rows * D - 16 * p.rows) / (8 * std::max(p.rows, 1))) / 32 * 32;
    p.keys_per_split = std::max(32, std::min(1024, kps));
  } else {
    // one wave per 16-row block, 1, 2 or 4 waves per work-group
    p.row_blocks = blocks16 <= 1 ? 1 : (blocks16 == 2 ? 2 : 4);
    p.row_groups = (blocks16 + p.row_blocks - 1) / p.row_blocks;
    p.rows_padded = p.row_groups * p.row_blocks * 16;
    // A work-group of 4 row blocks (8 waves in two key groups) holds a
    // 128 KB LDS ring, one per compute unit; smaller ones (1-2 waves) hold
    // 48 KB, three per unit.  Aim for that many work-groups per unit on 256
    // units, all resident at once; at least one 32-key tile per split.  Small work-groups over long caches split four times
    // finer: the splits are planned for the capacity, so with ragged
    // sequence lengths the longest sequence would otherwise stream its keys
    // through few work-groups, each bound by memory latency.
    const long long pairs = (long long)B * Hkv * p.row_groups;
    const long long target = p.row_blocks == 4 ? 256 : (capacity >= 8192 ? 3072 : 768);
    long long nsplit = std::max(1LL, (target + pairs - 1) / pairs);
    long long kps = (capacity + nsplit - 1) / nsplit;
    kps = std::max((long long)kTile, (kps + kTile - 1) / kTile * kTile);
    p.keys_per_split = (int)kps;
  }
  p.nsplit = std::max(1, (capacity + p.keys_per_split - 1) / p.keys_per_split);
  p.workspace_bytes = (size_t)B * Hkv * p.nsplit * p.rows_padded * ((size_t)D + 1) * sizeof(float);
  return p;
}

hipError_t launch_verify(const VerifyArgs& a, const VerifyPlan& p, int dtype, hipStream_t st) {
  const bool paged = a.page_table != nullptr;
  hipError_t e;
  if (dtype == 0) {
    const size_t lds = (size_t)p.rows * p.keys_per_split * 8 + (size_t)p.rows * 16 +
                       (size_t)p.rows * a.D * 4;
    dim3 grid(p.nsplit, a.Hkv, a.B);
    if (paged)
      hipLaunchKernelGGL(verify_split_f32<true>, grid, dim3(256), lds, st, a, p.keys_per_split,
                         p.nsplit, p.rows_padded);
    else
      hipLaunchKernelGGL(verify_split_f32<false>, grid, dim3(256), lds, st, a, p.keys_per_split,
                         p.nsplit, p.rows_padded);
    e = hipGetLastError();
  } else if (a.D == 128) {
    e = paged ? dispatch_rb<128, true>(a, p, st) : dispatch_rb<128, false>(a, p, st);
  } else {
    e = paged ? dispatch_rb<64, true>(a, p, st) : dispatch_rb<64, false>(a, p, st);
  }
  if (e != hipSuccess) return e;
  if (dtype != 0 && p.nsplit == 1) return hipSuccess;   // the split kernel wrote out / lse
  hipLaunchKernelGGL(verify_merge, dim3((p.rows + 3) / 4, a.Hkv * a.B), dim3(256), 0, st, a,
                     p.keys_per_split, p.nsplit, p.rows_padded, paged ? 1 : 0);
  return hipGetLastError();
}

}  // namespace sd
