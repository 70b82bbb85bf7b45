// Verification attention of the drafted block over the KV cache (SpecFLASH
// Sec. 3.1: the target scores all K drafted tokens in one parallel pass).
//
// The work is HBM-bound: every key / value of the cache is read once for
// all k * g query rows that share a KV head (k block positions times g
// grouped query heads), so the design keeps those rows resident and streams
// the cache.
//
// Kernel 1 (stream): a fixed grid sized to the device.  All (sequence, KV
//   head, row group) pairs form one list of 32-key tiles; each work-group
//   takes an equal contiguous range of it, so ragged sequence lengths stay
//   balanced to a tile.  A work-group holds up to 64 query rows (one wave
//   per 16-row block) and streams its tiles HBM -> LDS by the
//   global_load_lds DMA into a ring shared by its waves; per tile a wave
//     - computes S^T = K Q^T on bf16 matrix cores from K fragments in LDS,
//       so that every lane holds scores of exactly one query row (column c
//       of the accumulator);
//     - runs the online softmax in fp32 (base-2 exponent, masked by the
//       causal limit kv_len - k + j of its row on tail tiles only);
//     - accumulates O^T += V^T P^T, reading V^T fragments from LDS with the
//       transposing ds_read_b64_tr_b16, and feeding P as a bf16 hi + lo pair
//       (P = hi + lo to ~2^-16 relative), which keeps the result within the
//       float tolerance of the fp32 reference without converting V.
//   Work-groups of 4 row blocks run 8 waves: two key groups of 4 take
//   alternate tiles of one deep ring.  Wherever its range moves to the next
//   pair, a work-group writes the normalised partial (o, lse) of the
//   finished segment.
// Kernel 2 (merge): finds the partials of each pair from the same tile
//   arithmetic, combines them with the log-sum-exp rule and writes out / lse
//   in the caller's [B, k, Hq] layout.
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

// bf16 stream kernel configuration by 16-row blocks per work-group (1, 2
// or 4): key groups (waves = blocks x key groups), ring slots of one tile
// (16 KB for D = 128) and work-groups per compute unit
struct StreamCfg {
  int kg, nbuf, per_cu;
};
constexpr StreamCfg stream_cfg(int row_blocks) {
  return row_blocks == 4 ? StreamCfg{2, 8, 1} : StreamCfg{1, 4, 2};
}

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

// ----------------------------------------------------------- bf16 stream
// All (sequence, KV head, row group) pairs of a call form one list of 32-key
// tiles, in the order sequence b, then x = KV head * row_groups + row group,
// then the tiles t of sequence b:
//   n = cum(b) X + x nt(b) + t,  nt(b) = ceil(kv_len[b] / 32),
//   cum(b) = nt(0) + ... + nt(b - 1),  X = Hkv row_groups,  T = cum(B) X.
// Work-group w of G owns the tiles [T w / G, T (w + 1) / G), so the work
// is balanced to a tile however ragged the lengths are; the bounds come
// from kv_len on the device (the host sizes nothing by the lengths).
// Where its range changes pair, a work-group writes the partial (o, lse)
// of the finished segment to slot (pair + w) KG + key group: along the
// tile order both the pair and w only grow, so pair + w is distinct for
// every segment, and P + G slots per key group suffice.

typedef const __attribute__((address_space(4))) int32_t cint32;   // scalar loads

struct TileCursor {
  int b, x, t;   // sequence, KV head * row_groups + row group, tile
  int nt, L;     // tiles and length of sequence b
};

// length of sequence b as a scalar load (no vector-memory counter use)
__device__ __forceinline__ int seq_len_s(const VerifyArgs& a, int b, int cap) {
  return min(max(((cint32*)a.kv_len)[b], 0), cap);
}

// cum(b_end) (tiles of sequences before b_end, times X) over the first
// b_end sequences; every lane of the wave gets the same value
__device__ __forceinline__ int tiles_before(const VerifyArgs& a, int X, int cap, int b_end) {
  const int lane = threadIdx.x & 63;
  int sum = 0;
  for (int b0 = 0; b0 < b_end; b0 += 64) {
    const int b = b0 + lane;
    int v = 0;
    if (b < b_end) v = (min(max(a.kv_len[b], 0), cap) + 31) >> 5;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    sum += v;
  }
  return sum * X;
}

// cursor of tile n (0 <= n < T); wave-uniform
__device__ __forceinline__ TileCursor locate(const VerifyArgs& a, int X, int cap, int n) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  TileCursor cu{0, 0, 0, 0, 0};
  for (int b0 = 0; b0 < a.B; b0 += 64) {
    const int b = b0 + lane;
    const int L = b < a.B ? min(max(a.kv_len[b], 0), cap) : 0;
    const int span = ((L + 31) >> 5) * X;
    int incl = span;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    const unsigned long long hit = __ballot(base + incl > n);
    if (hit != 0ull) {
      const int f = __builtin_ctzll(hit);
      const int Lf = __shfl(L, f, 64);
      const int ex = __shfl(incl - span, f, 64);   // tiles before sequence b0 + f
      cu.b = b0 + f;
      cu.L = Lf;
      cu.nt = (Lf + 31) >> 5;
      const int rem = n - base - ex;
      cu.x = rem / cu.nt;
      cu.t = rem - cu.x * cu.nt;
      return cu;
    }
    base += __shfl(incl, 63, 64);
  }
  return cu;   // n >= T: not reached
}

// Tile bookkeeping from one load of kv_len when B <= 64 (lane b holds
// sequence b): the total T and the cursors of tiles n_a and n_b, where
// n_a = T * wg / G and n_b = min(n_a + off_b, T * (wg + 1) / G - 1).
// Returns false (nothing computed) when B > 64.
struct TileStart {
  int T, n0, n1;
  TileCursor ca, cb;
};

__device__ __forceinline__ bool tile_start_small(const VerifyArgs& a, int X, int cap, int wg, int G,
                                                 int off_b, TileStart* ts) {
  if (a.B > 64) return false;
  const int lane = threadIdx.x & 63;
  const int L = lane < a.B ? min(max(a.kv_len[lane], 0), cap) : 0;
  const int nt = (L + 31) >> 5;
  const int span = nt * X;
  int incl = span;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  const int T = __shfl(incl, 63, 64);
  ts->T = T;
  ts->n0 = (int)((long long)T * wg / G);
  ts->n1 = (int)((long long)T * (wg + 1) / G);
  if (ts->n0 >= ts->n1) return true;
  auto find = [&](int n) {
    TileCursor cu;
    const unsigned long long hit = __ballot(incl > n);
    const int f = __builtin_ctzll(hit);
    cu.b = f;
    cu.L = __shfl(L, f, 64);
    cu.nt = (cu.L + 31) >> 5;
    const int rem = n - __shfl(incl - span, f, 64);
    cu.x = rem / cu.nt;
    cu.t = rem - cu.x * cu.nt;
    return cu;
  };
  ts->ca = find(ts->n0);
  ts->cb = find(min(ts->n0 + off_b, ts->n1 - 1));
  return true;
}

// the same cursor held in scalar registers
__device__ __forceinline__ TileCursor uniform(TileCursor cu) {
  cu.b = __builtin_amdgcn_readfirstlane(cu.b);
  cu.x = __builtin_amdgcn_readfirstlane(cu.x);
  cu.t = __builtin_amdgcn_readfirstlane(cu.t);
  cu.nt = __builtin_amdgcn_readfirstlane(cu.nt);
  cu.L = __builtin_amdgcn_readfirstlane(cu.L);
  return cu;
}

// next tile in the global order; the caller never steps past the last tile
__device__ __forceinline__ void advance(const VerifyArgs& a, int X, int cap, TileCursor& cu) {
  if (++cu.t < cu.nt) return;
  cu.t = 0;
  if (++cu.x < X) return;
  cu.x = 0;
  do {
    ++cu.b;
    cu.L = cu.b < a.B ? seq_len_s(a, cu.b, cap) : 0;
    cu.nt = (cu.L + 31) >> 5;
  } while (cu.nt == 0 && cu.b < a.B);
}

// One work-group = NW = NWR x KG waves: NWR 16-row blocks of one pair, KG
// key groups taking alternate tiles.  Tiles go HBM -> LDS by the
// global_load_lds DMA into a ring of NBUF slots, NBUF - KG tiles ahead of
// the compute.  Each key row keeps its 16-byte pieces XOR-swizzled by
// lds_swizzle(key), so the K-fragment reads (16 keys x one piece) and the
// transposed V reads (4 keys x 8 bytes per 16 lanes) are free of bank
// conflicts.  Per tile a wave does 8 + 16 matrix-core ops and little else:
// the causal mask is applied only on the tail tile of a sequence, the
// running maximum is raised (and O, l rescaled) only when a row's scores
// exceed it by more than 2^8 (the stale maximum is exact for the final
// o = O / l; p stays below 256).
template <int D, int NWR, int KG, int NBUF, bool PAGED>
__global__ __launch_bounds__(NWR * KG * 64) void verify_stream_bf16(VerifyArgs a, int G,
                                                                    int row_groups) {
  constexpr int NW = NWR * KG;
  constexpr int TK = kTile;
  constexpr int DC = D / 32;                   // 32-channel K slices (QK^T)
  constexpr int DB = D / 16;                   // 16-channel output blocks (PV)
  constexpr int PK = D / 8;                    // 16-byte pieces per key row
  constexpr int ROW_BYTES = D * 2;
  constexpr int HALF_BYTES = TK * ROW_BYTES;   // K (or V) part of a slot
  constexpr int BUF_BYTES = 2 * HALF_BYTES;
  constexpr int DMA_PER_HALF = TK * PK / 64;   // 64-lane copies per K (or V) tile
  constexpr int DMA_PER_WAVE = 2 * DMA_PER_HALF / NW;   // per tile
  constexpr int ROWS_WG = NWR * 16;
  static_assert((2 * DMA_PER_HALF) % NW == 0, "tile copy must split evenly");
  static_assert(TK == 32, "one P V step per tile");
  static_assert(NBUF >= 2 * KG + 1 && (NBUF - 2 * KG) * DMA_PER_WAVE < 64,
                "ring depth and vmcnt range");
  constexpr float kRescale = 8.f;              // log2 headroom before rescaling
  __shared__ __align__(16) unsigned char ring[NBUF][BUF_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63, G4 = lane >> 4, c = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w % NWR, kgrp = w / NWR;      // row block, key group
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int X = a.Hkv * row_groups;
  const int cap = PAGED ? a.max_pages * 16 : a.Lmax;
  // Logical work-group: the two low 3-bit fields of the hardware index
  // swapped (grids of 64k work-groups).  Consecutive hardware work-groups
  // go to different XCDs; with this order the work-groups that stream the
  // same key range of 8 consecutive pairs (the 8 KV heads of a sequence,
  // whose 256-byte slices share each cache row) sit on 8 different XCDs,
  // which streams about 5% faster than giving one XCD the whole row.
  const int hw = blockIdx.x;
  const int wg = (gridDim.x & 63) == 0 ? ((hw & ~63) | ((hw & 7) << 3) | ((hw >> 3) & 7)) : hw;
  TileStart ts;
  if (!tile_start_small(a, X, cap, wg, G, kgrp, &ts)) {
    ts.T = tiles_before(a, X, cap, a.B);
    ts.n0 = (int)((long long)ts.T * wg / G);
    ts.n1 = (int)((long long)ts.T * (wg + 1) / G);
    if (ts.n0 < ts.n1) {
      ts.ca = locate(a, X, cap, ts.n0);
      ts.cb = locate(a, X, cap, min(ts.n0 + kgrp, ts.n1 - 1));
    }
  }
  const int n0 = __builtin_amdgcn_readfirstlane(ts.n0);
  const int n1 = __builtin_amdgcn_readfirstlane(ts.n1);
  if (n0 >= n1) return;
  const int last = n1 - 1;

  // per-lane constants of the copies: copy i of this wave (ii = w *
  // DMA_PER_WAVE + i) covers half ii / DMA_PER_HALF (K or V) and pieces
  // P = (ii % DMA_PER_HALF) * 64 + lane: key P / PK, LDS slot P % PK holding
  // global piece slot ^ lds_swizzle(key).  The element offset of a copy is
  // a uniform tile base plus this per-lane part.
  int ckey[DMA_PER_WAVE];
  uint32_t clane[DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < DMA_PER_WAVE; ++i) {
    const int ii = w * DMA_PER_WAVE + i;
    const int P = (ii % DMA_PER_HALF) * 64 + lane;
    const int key = P / PK;
    const int piece = ((P % PK) ^ lds_swizzle<PK>(key)) * 8;
    ckey[i] = key;
    clane[i] = PAGED ? (uint32_t)((key & 15) * D + piece) : (uint32_t)(key * a.Hkv * D + piece);
  }
  const uint16_t* kbase = static_cast<const uint16_t*>(a.kc);
  const uint16_t* vbase = static_cast<const uint16_t*>(a.vc);
  // copies of the tile under cursor cu; keys past the sequence re-read its
  // last key (masked).  Page ids are scalar loads, so they do not count
  // against vmcnt.
  auto issue = [&](const TileCursor& cu, unsigned char* slot) {
    const int t0 = cu.t * TK;
    const int hk = cu.x / row_groups;
    const bool tail = t0 + TK > cu.L;
    int pg0 = 0, pg1 = 0;
    if constexpr (PAGED) {
      cint32* pt = (cint32*)(a.page_table + (size_t)cu.b * a.max_pages);
      const int lastp = (cu.L - 1) >> 4;
      pg0 = min(max((int)pt[min(t0 >> 4, lastp)], 0), a.num_pages - 1);
      pg1 = min(max((int)pt[min((t0 >> 4) + 1, lastp)], 0), a.num_pages - 1);
    }
    const size_t tbase = PAGED ? 0 : (((size_t)cu.b * a.Lmax + t0) * a.Hkv + hk) * D;
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const int ii = w * DMA_PER_WAVE + i;
      const int half = ii / DMA_PER_HALF;
      const int key = ckey[i];
      size_t off;
      if constexpr (PAGED) {
        uint32_t lo = clane[i];
        int pk = key >> 4;                     // page 0 or 1 of the tile
        if (tail && t0 + key > cu.L - 1) {     // re-read the last key
          const int t = cu.L - 1 - t0;
          lo = (uint32_t)((t & 15) * D) + (clane[i] & (uint32_t)(PK * 8 - 1));
          pk = t >> 4;
        }
        off = ((size_t)(pk ? pg1 : pg0) * a.Hkv + hk) * 16 * D + lo;
      } else {
        off = tbase + clane[i];
        if (tail && t0 + key > cu.L - 1)       // re-read the last key
          off -= (size_t)(t0 + key - (cu.L - 1)) * a.Hkv * D;
      }
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)((half ? vbase : kbase) + off),
                                       (lds_void*)(slot + half * HALF_BYTES + (ii % DMA_PER_HALF) * 1024),
                                       16, 0, 0);
    }
  };

  // per-lane LDS offsets of the fragment reads inside a slot, for the first
  // 16-key block; the swizzle depends on key % 16 only, so the second block
  // (+16 keys) is an immediate offset of the read
  uint32_t koff[DC];
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) koff[dc] = c * ROW_BYTES + (((dc * 4 + G4) ^ lds_swizzle<PK>(c)) * 16);
  // ds_read_b64_tr_b16: lane j of group G4 addresses key 4 G4 + j / 4 (+16)
  // at channels db * 16 + 4 (j % 4); lane c then receives 4 keys at channel
  // db * 16 + c
  uint32_t voff[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int key = 4 * G4 + (c >> 2);
    const int ch = db * 16 + 4 * (c & 3);
    voff[db] = HALF_BYTES + key * ROW_BYTES + (((ch >> 3) ^ lds_swizzle<PK>(key)) * 16) + (ch & 7) * 2;
  }

  // segment state of this wave: pair, query row, its B operand of
  // S^T = K Q^T, causal limit, running (max, sum, O^T)
  int cur_pair = -1;
  bool row_ok = false;
  int lim = -1, orow = 0, unmasked_end = 0;
  bf16x8 qf[DC];
  float m = -INFINITY, l = 0.f;
  floatx4 o[DB];
  // Scores stay raw (S = K Q^T); the scale enters the exponent as
  // exp2(S sl2 - m).  A negative scale is folded into the queries
  // (softmax(s q.k) = softmax(|s| (-q).k)), so sl2 >= 0 below.
  const bool neg_scale = a.scale_log2 < 0.f;
  const float sl2 = fabsf(a.scale_log2);

  auto start_segment = [&](const TileCursor& cu) {
    const int hk = cu.x / row_groups, rg = cu.x % row_groups;
    const int r = rg * ROWS_WG + wr * 16 + c;
    row_ok = r < R;
    Pack8 pk;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      pk.u = u32x4{0u, 0u, 0u, 0u};
      qf[dc] = pk.b;
    }
    lim = -1;
    if (row_ok) {
      const int j = r / g;
      const int h = hk * g + (r - j * g);
      orow = (cu.b * a.k + j) * a.Hq + h;
      const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.q) + (size_t)orow * D);
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        pk.u = src[dc * 4 + G4];
        if (neg_scale) pk.u ^= u32x4{0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u};
        qf[dc] = pk.b;
      }
      lim = cu.L - a.k + j;                    // last visible key of this row
    }
    unmasked_end = cu.L - a.k;                 // every row sees keys 0 .. L - k
    m = -INFINITY;
    l = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = floatx4{0.f, 0.f, 0.f, 0.f};
  };
  auto flush = [&]() {
    const float lsum = wave_sum_across_groups(l);
    if (!row_ok) return;
    const size_t prow = ((size_t)(cur_pair + wg) * KG + kgrp) * ROWS_WG + wr * 16 + c;
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<floatx4*>(a.part_o + prow * D + db * 16 + 4 * G4) = o[db] * inv;
    if (G4 == 0) a.part_lse[prow] = lsum > 0.f ? m + log2f(lsum) : -INFINITY;
  };

  auto compute = [&](int t0, const unsigned char* slot) {
    const uint32_t sb = lds_addr(slot);
    u32x4 kr[2][DC];
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      kr[0][dc] = lds_read_b128_off<0>(sb + koff[dc]);
      kr[1][dc] = lds_read_b128_off<16 * ROW_BYTES>(sb + koff[dc]);
    }
    lds_wait();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) tie(kr[kb][dc]);
    // V^T fragments for P V, issued now so they overlap the scores
    u32x2 vr[2][DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      vr[0][db] = lds_read_tr16_b64_off<0>(sb + voff[db]);
      vr[1][db] = lds_read_tr16_b64_off<16 * ROW_BYTES>(sb + voff[db]);
    }

    // S^T = K Q^T: lane holds S[row c][key t0 + kb*16 + 4 G4 + i] (raw)
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
      for (int i = 0; i < 4; ++i) x[kb * 4 + i] = acc[i];
    }

    // Online softmax with a lazily raised maximum.  Each lane forms the
    // exponents y = S sl2 - m of its 8 scores, taken before the causal mask
    // (so their largest bounds the masked ones from above), and checks the
    // largest against kRescale (+inf before the first raise, m = -inf);
    // only when some lane passes it are the row maxima formed across the
    // row's four lanes and m raised.  m may so exceed the masked tile's true
    // maximum, which leaves o = O / l and lse = m + log2 l unchanged, and P
    // (bf16 hi + lo, the fp32 exponent range) neither overflows nor loses
    // precision.
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = fmaf(x[e], sl2, -m);
    const float ly = fmaxf(fmaxf(fmaxf(y[0], y[1]), fmaxf(y[2], y[3])),
                           fmaxf(fmaxf(y[4], y[5]), fmaxf(y[6], y[7])));
    if (__ballot(ly > kRescale) != 0ull) {
      const float lm = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                             fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
      const float mnew = fmaxf(m, wave_max_across_groups(lm) * sl2);
      const float alpha = (m == -INFINITY) ? 0.f : fast_exp2(m - mnew);   // O, l are still 0 before the first raise
      l *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
      m = mnew;
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = fmaf(x[e], sl2, -m);
    }
    float pv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pv[e] = fast_exp2(y[e]);
    if (t0 + TK - 1 > unmasked_end) {          // tail tile: causal mask
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int t = t0 + (e >> 2) * 16 + 4 * G4 + (e & 3);
        if (t > lim) pv[e] = 0.f;
      }
    }
    // P = hi + lo: hi the bf16 truncation (a mask of the fp32 bits), lo the
    // exact remainder (|lo| < 2^-7 p) rounded to bf16, so P is kept to
    // 2^-16 of p
    Pack8 phk, plk;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const uint32_t b0 = __float_as_uint(pv[e]), b1 = __float_as_uint(pv[e + 1]);
      psum += pv[e] + pv[e + 1];
      phk.u[e / 2] = __builtin_amdgcn_perm(b1, b0, 0x07060302u);   // high halves of b0 | b1
      plk.b[e] = float_to_bf16(pv[e] - __uint_as_float(b0 & 0xffff0000u));
      plk.b[e + 1] = float_to_bf16(pv[e + 1] - __uint_as_float(b1 & 0xffff0000u));
    }
    const bf16x8 ph = phk.b, pl = plk.b;
    l += psum;

    // O^T += V^T P^T.  The product's K index runs over keys {4G4..4G4+3,
    // 16+4G4..16+4G4+3}, the order in which the score accumulator handed
    // this lane its P values; accumulator element i of block db is channel
    // db*16 + 4 G4 + i of row c.
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

  // Every step issues KG tiles (past the range it re-reads the last one,
  // which is still cached), so exactly (NBUF - 2 KG) tiles' copies are newer
  // than the step's own tiles at each wait, and the wait covers precisely
  // the tiles about to be read; the barrier also frees the slots of the
  // previous step for refilling.  The tile reads are asm, so the compiler
  // adds no waits of its own between them and the copies.  A new segment
  // (query loads, partial stores) drains this wave's memory counter first,
  // so the counted waits only ever see copies.
  TileCursor ic = uniform(ts.ca);              // issue cursor at tile in
  int in = n0;
  TileCursor cc = uniform(ts.cb);              // compute cursor at tile cn
  int cn = n0 + kgrp;
  const int nsteps = (n1 - n0 + KG - 1) / KG;
#pragma unroll 1
  for (int i = 0; i < NBUF - KG; ++i) {
    issue(ic, ring[i]);
    if (in < last) {
      advance(a, X, cap, ic);
      ++in;
    }
  }
#pragma unroll 1
  for (int s = 0; s < nsteps; ++s) {
    wait_vm_then_barrier<(NBUF - 2 * KG) * DMA_PER_WAVE>();
#pragma unroll
    for (int j = 0; j < KG; ++j) {
      issue(ic, ring[(s * KG + NBUF - KG + j) % NBUF]);
      if (in < last) {
        advance(a, X, cap, ic);
        ++in;
      }
    }
    if (cn <= last) {                          // wave-uniform
      const int pair = cc.b * X + cc.x;
      if (pair != cur_pair) {
        if (cur_pair >= 0) flush();
        start_segment(cc);
        cur_pair = pair;
        __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
      }
      compute(cc.t * TK, ring[(s * KG + kgrp) % NBUF]);
#pragma unroll
      for (int j = 0; j < KG; ++j) {
        if (cn < last) {
          advance(a, X, cap, cc);
        }
        ++cn;
      }
    }
  }
  // no copy may still be writing this work-group's LDS when it exits
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
  if constexpr (KG == 2) {
    // When both key groups end on the same pair, group 1 hands its (max,
    // sum, O) to group 0 through the ring and one combined partial is
    // written (slot key group 0); otherwise each group writes its own.
    __syncthreads();                           // every wave is done with the ring
    int* xpair = reinterpret_cast<int*>(&ring[0][0]);
    floatx4* xo = reinterpret_cast<floatx4*>(&ring[0][0] + 256);
    float2* xml = reinterpret_cast<float2*>(&ring[0][0] + 256 + NWR * DB * 64 * 16);
    if (lane == 0) xpair[w] = cur_pair;
    __syncthreads();
    const bool joint = cur_pair >= 0 && xpair[wr] == xpair[NWR + wr];   // wave-uniform
    if (kgrp == 1 && joint) {
      const float lsum = wave_sum_across_groups(l);
#pragma unroll
      for (int db = 0; db < DB; ++db) xo[(wr * DB + db) * 64 + lane] = o[db];
      xml[wr * 64 + lane] = make_float2(m, lsum);
    }
    __syncthreads();
    if (kgrp == 1) {
      if (!joint && cur_pair >= 0) flush();
      return;
    }
    if (joint) {
      const float2 ml = xml[wr * 64 + lane];
      const float mn = fmaxf(m, ml.x);
      const float f0 = m == -INFINITY ? 0.f : fast_exp2(m - mn);
      const float f1 = ml.x == -INFINITY ? 0.f : fast_exp2(ml.x - mn);
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] = o[db] * f0 + xo[(wr * DB + db) * 64 + lane] * f1;
      // l is per lane until flush sums it over the row; the partner's sum
      // is added on one lane of the row only
      l = l * f0 + (G4 == 0 ? ml.y * f1 : 0.f);
      m = mn;
    }
  }
  if (cur_pair >= 0) flush();
}

// ----------------------------------------------------------- fp32 split
// fp32 inputs: scores, softmax and P V run in float64, so the result keeps
// full fp32 accuracy even when large scores make the softmax sensitive to
// rounding.  One work-group per (key split, KV head, sequence), splits
// fastest on a 1-D grid, with short splits, so the
// work spreads over many compute units.  The block's queries and the
// split's key and value rows are staged in LDS with coalesced loads (rows
// padded by one float, so that lanes reading the same channel of
// consecutive rows hit distinct banks); the split's scores sit in LDS; one
// wave per row forms the softmax statistics; threads over (row, channel)
// accumulate P V.
template <bool PAGED>
__global__ __launch_bounds__(256) void verify_split_f32(VerifyArgs a, int keys_per_split,
                                                        int nsplit, int rows_padded) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int D = a.D, DS = D + 1;
  const int split = (int)(blockIdx.x % (unsigned)nsplit);
  const int pair = (int)(blockIdx.x / (unsigned)nsplit);
  const int hk = pair % a.Hkv;
  const int b = pair / a.Hkv;
  const int L = seq_len(a, b, PAGED);
  const int k0 = split * keys_per_split;
  if (k0 >= L) return;
  const int nk = min(L, k0 + keys_per_split) - k0;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int tid = threadIdx.x;

  double* ss = reinterpret_cast<double*>(smem);         // [R][keys_per_split]
  double* st = ss + (size_t)R * keys_per_split;         // [R][2]: max, sum
  float* qs = reinterpret_cast<float*>(st + 2 * R);     // [R][D + 1]
  float* ks = qs + (size_t)R * DS;                       // [keys_per_split][D + 1]
  float* vs = ks + (size_t)keys_per_split * DS;          // [keys_per_split][D + 1]
  const float* qg = static_cast<const float*>(a.q);
  const float* kg = static_cast<const float*>(a.kc);
  const float* vg = static_cast<const float*>(a.vc);
  {
    // rows start at multiples of D floats: 16-byte loads when the bases
    // are 16-byte aligned, else 4-byte loads (fp32 needs only the latter)
    float* const qd[1] = {qs};
    const float* const qsrc[1] = {qg};
    float* const kvd[2] = {ks, vs};
    const float* const kvsrc[2] = {kg, vg};
    auto qrow = [&](int r) {
      const int j = r / g, h = hk * g + (r - j * g);
      return (((size_t)b * a.k + j) * a.Hq + h) * D;
    };
    auto kvrow = [&](int tt) { return kv_offset<PAGED>(a, b, hk, k0 + tt, D); };
    if (((reinterpret_cast<uintptr_t>(qg) | reinterpret_cast<uintptr_t>(kg) | reinterpret_cast<uintptr_t>(vg)) &
         15) == 0) {
      stage_rows<4, 1, 4>(qd, DS, qsrc, qrow, R, D);
      stage_rows<4, 2, 4>(kvd, DS, kvsrc, kvrow, nk, D);
    } else {
      stage_rows<8, 1, 1>(qd, DS, qsrc, qrow, R, D);
      stage_rows<8, 2, 1>(kvd, DS, kvsrc, kvrow, nk, D);
    }
  }
  __syncthreads();
  const double scale = (double)a.scale;
  // thread i: row i / nk, key i % nk (consecutive lanes take consecutive keys)
  for (int i = tid; i < nk * R; i += blockDim.x) {
    const int r = i / nk, tt = i - r * nk;
    const int j = r / g;
    double s = -INFINITY;
    if (k0 + tt <= L - a.k + j) {
      const float* qr = qs + r * DS;
      const float* kr = ks + tt * DS;
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
    const int r = i / D, e = i - r * D;
    const double sum = st[2 * r + 1];
    const double* pr = ss + (size_t)r * keys_per_split;
    double acc = 0.0;
    // a zero weight adds nothing, even against a non-finite value
#pragma unroll 8
    for (int tt = 0; tt < nk; ++tt) {
      const double p = pr[tt];
      const double v = (double)vs[tt * DS + e];
      acc = fma(p, p != 0.0 ? v : 0.0, acc);
    }
    a.part_o[(base + r) * D + e] = sum > 0.0 ? (float)(acc / sum) : 0.f;
    if (e == 0)
      a.part_lse[base + r] =
          sum > 0.0 ? (float)((st[2 * r] + log(sum)) * 1.4426950408889634) : -INFINITY;
  }
}

// ---------------------------------------------------------------- merge
// One wave per output row of one (sequence, KV head).  The splits are taken
// 32 at a time: lanes 0..31 load their split's lse while each half-wave
// loads the partial outputs of 16 splits (4 channels per lane), all in one
// round of memory accesses; the chunk's weights 2^(lse - max) then rescale
// a running sum as in the online softmax.  Every shuffle runs on all lanes.
// Grid (sequence x KV head, rows / 4).
__global__ __launch_bounds__(256) void verify_merge(VerifyArgs a, int keys_per_split,
                                                    int nsplit, int rows_padded, int paged) {
  const int pair = blockIdx.x;
  const int hk = pair % a.Hkv;
  const int b = pair / a.Hkv;
  const int D = a.D;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.y * 4 + w;
  if (r >= R) return;
  const int L = seq_len(a, b, paged != 0);
  const int nvalid = min(nsplit, (L + keys_per_split - 1) / keys_per_split);
  const size_t base = (size_t)pair * nsplit * rows_padded + r;
  const int half = lane >> 5, d4 = lane & 31;
  const bool active = d4 < D / 4;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float mx = -INFINITY, wsum = 0.f;
  for (int s0 = 0; s0 < nvalid; s0 += 32) {
    const int n = min(32, nvalid - s0);
    const float ls = lane < n ? a.part_lse[base + (size_t)(s0 + lane) * rows_padded] : -INFINITY;
    floatx4 po[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int j = 2 * i + half;
      po[i] = floatx4{0.f, 0.f, 0.f, 0.f};
      if (j < n && active)
        po[i] = *reinterpret_cast<const floatx4*>(a.part_o + (base + (size_t)(s0 + j) * rows_padded) * D + d4 * 4);
    }
    float cm = ls;
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, 64));
    const float nm = fmaxf(mx, __shfl(cm, 0, 64));
    if (nm == -INFINITY) continue;             // no key in any split so far (uniform)
    const float keep = mx == -INFINITY ? 0.f : exp2f(mx - nm);
    const float wl = ls == -INFINITY ? 0.f : exp2f(ls - nm);
    float ws = wl;
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) ws += __shfl_xor(ws, off, 64);
    wsum = wsum * keep + __shfl(ws, 0, 64);
    acc = acc * keep;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc += __shfl(wl, 2 * i + half, 64) * po[i];
    mx = nm;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) acc[e] += __shfl_xor(acc[e], 32, 64);
  const int j = r / g;
  const int h = hk * g + (r - j * g);
  const size_t orow = ((size_t)b * a.k + j) * a.Hq + h;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  if (half == 0 && active) *reinterpret_cast<floatx4*>(a.out + orow * D + d4 * 4) = acc * inv;
  if (a.lse != nullptr && lane == 0)
    a.lse[orow] = wsum > 0.f ? (mx + log2f(wsum)) * kLn2 : -INFINITY;
}

// -------------------------------------------------------- stream merge
// One wave per output row of one pair (sequence b, x = KV head * row_groups
// + row group).  The pair's tiles [U, U + nt(b)) were spread over work-
// groups owner(U) .. owner(U + nt - 1), owner(n) = floor(((n + 1) G - 1) /
// T); key group kg of work-group w wrote slot (pair + w) KG + kg if one of
// its tiles (every KG-th from the range start) falls in the pair.  The
// candidate partials are taken 32 at a time: lanes 0..31 find their slots
// and load their lse while each half-wave loads the outputs of 16 of them
// (4 channels per lane), in one round of memory accesses; the chunk's weights 2^(lse - max)
// then rescale a running sum as in the online softmax.  Every shuffle runs
// on all lanes.  Grid (pairs, ceil(rows per pair / 4)).
__global__ __launch_bounds__(256) void verify_stream_merge(VerifyArgs a, int G, int row_groups,
                                                           int KG, int rows_wg, int paged) {
  const int pair = blockIdx.x;
  const int X = a.Hkv * row_groups;
  const int b = pair / X, x = pair - b * X;
  const int hk = x / row_groups, rg = x - hk * row_groups;
  const int D = a.D;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = blockIdx.y * 4 + w;           // row within the pair
  const int r = rg * rows_wg + lr;
  if (lr >= rows_wg || r >= R) return;
  const int cap = paged ? a.max_pages * 16 : a.Lmax;
  int T, U, nt;
  if (a.B <= 64) {                             // one load: lane b' holds sequence b'
    const int Lb = lane < a.B ? min(max(a.kv_len[lane], 0), cap) : 0;
    const int span = ((Lb + 31) >> 5) * X;
    int incl = span;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    T = __shfl(incl, 63, 64);
    nt = (__shfl(Lb, b, 64) + 31) >> 5;
    U = __shfl(incl - span, b, 64) + x * nt;
  } else {
    T = tiles_before(a, X, cap, a.B);
    nt = (seq_len(a, b, paged != 0) + 31) >> 5;
    U = tiles_before(a, X, cap, b) + x * nt;
  }
  const int half = lane >> 5, d4 = lane & 31;
  const bool active = d4 < D / 4;
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float mx = -INFINITY, wsum = 0.f;
  if (nt > 0) {
    // range start of work-group v: floor(T v / G) = qt v + floor(rt v / G)
    const unsigned qt = (unsigned)T / (unsigned)G, rt = (unsigned)T % (unsigned)G;
    auto wstart = [&](int v) { return (int)(qt * (unsigned)v + (rt * (unsigned)v) / (unsigned)G); };
    auto owner = [&](int n) { return (int)((((long long)n + 1) * G - 1) / T); };
    const int wf = owner(U), wl = owner(U + nt - 1);
    const int ncand = (wl - wf + 1) * KG;
    for (int c0 = 0; c0 < ncand; c0 += 32) {
      const int n = min(32, ncand - c0);
      // lane i < n: slot of candidate c0 + i (key group kg of work-group
      // wv), or -1 when that key group has no tile of the pair
      int sl = -1;
      if (lane < n) {
        const int cand = c0 + lane;
        const int wv = wf + cand / KG, kg = cand - (cand / KG) * KG;
        const int s0 = wstart(wv), s1 = wstart(wv + 1);
        const int lo = max(U, s0), hi = min(U + nt, s1);
        const int first = s0 + kg + (lo > s0 + kg ? (lo - s0 - kg + KG - 1) / KG * KG : 0);
        if (first < hi) sl = (pair + wv) * KG + kg;
        if (KG == 2 && kg == 1 && sl >= 0) {
          // both groups' last tiles in this pair: one combined partial
          const int last0 = s0 + (s1 - 1 - s0) / 2 * 2;
          const int last1 = s0 + 1 + (s1 - 2 - s0) / 2 * 2;
          if (last0 >= U && last0 < U + nt && last1 >= U && last1 < U + nt) sl = -1;
        }
      }
      const float ls = sl >= 0 ? a.part_lse[(size_t)sl * rows_wg + lr] : -INFINITY;
      floatx4 po[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int sj = __shfl(sl, 2 * i + half, 64);
        po[i] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (sj >= 0 && active)
          po[i] = *reinterpret_cast<const floatx4*>(a.part_o + ((size_t)sj * rows_wg + lr) * D + d4 * 4);
      }
      float cm = ls;
#pragma unroll
      for (int off = 16; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, 64));
      const float nm = fmaxf(mx, __shfl(cm, 0, 64));
      if (nm == -INFINITY) continue;           // no key in any partial so far (uniform)
      const float keep = mx == -INFINITY ? 0.f : exp2f(mx - nm);
      const float wl8 = ls == -INFINITY ? 0.f : exp2f(ls - nm);
      float ws = wl8;
#pragma unroll
      for (int off = 16; off > 0; off >>= 1) ws += __shfl_xor(ws, off, 64);
      wsum = wsum * keep + __shfl(ws, 0, 64);
      acc = acc * keep;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc += __shfl(wl8, 2 * i + half, 64) * po[i];
      mx = nm;
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) acc[e] += __shfl_xor(acc[e], 32, 64);
  const int j = r / g;
  const int h = hk * g + (r - j * g);
  const size_t orow = ((size_t)b * a.k + j) * a.Hq + h;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  if (half == 0 && active) {
    const floatx4 o = acc * inv;
    if (a.out_bf16 != nullptr) {
      Pack8 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk.b[e] = float_to_bf16(o[e]);
      *reinterpret_cast<u32x2*>(a.out_bf16 + orow * D + d4 * 4) = u32x2{pk.u[0], pk.u[1]};
    } else {
      *reinterpret_cast<floatx4*>(a.out + orow * D + d4 * 4) = o;
    }
  }
  if (a.lse != nullptr && lane == 0)
    a.lse[orow] = wsum > 0.f ? (mx + log2f(wsum)) * kLn2 : -INFINITY;
}

template <int D, int NWR, int KG, int NBUF, bool PAGED>
hipError_t launch_stream(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  hipLaunchKernelGGL((verify_stream_bf16<D, NWR, KG, NBUF, PAGED>), dim3(p.stream_wgs),
                     dim3(NWR * KG * 64), 0, st, a, p.stream_wgs, p.row_groups);
  return hipGetLastError();
}

template <int D, bool PAGED>
hipError_t dispatch_rb(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  switch (p.row_blocks) {
    case 1: return launch_stream<D, 1, stream_cfg(1).kg, stream_cfg(1).nbuf, PAGED>(a, p, st);
    case 2: return launch_stream<D, 2, stream_cfg(2).kg, stream_cfg(2).nbuf, PAGED>(a, p, st);
    default: return launch_stream<D, 4, stream_cfg(4).kg, stream_cfg(4).nbuf, PAGED>(a, p, st);
  }
}

}  // namespace

VerifyPlan plan_verify(int B, int k, int Hq, int Hkv, int D, int capacity, int dtype, int cus) {
  VerifyPlan p{};
  p.g = Hq / Hkv;
  p.rows = k * p.g;
  p.capacity = capacity;
  p.ok = true;
  const int blocks16 = (p.rows + 15) / 16;
  if (dtype == 0) {  // fp32 path: all rows in one work-group, splits by capacity
    p.row_blocks = blocks16;
    p.row_groups = 1;
    p.rows_padded = p.rows;
    // short splits (64 keys at most) so that the grid spreads over the
    // device; fp32 queries and the split's keys and values (rows padded by
    // one float), fp64 scores and row statistics within 64 KB of LDS
    int kps = 64;
    while (kps > 8 && (size_t)p.rows * (D + 1) * 4 + (size_t)2 * kps * (D + 1) * 4 + (size_t)8 * p.rows * kps +
                          16 * (size_t)p.rows > 65536)
      kps /= 2;
    // shorter splits (16 keys at least) while the grid would leave compute
    // units idle: a work-group's scores and P V are serial float64 chains,
    // so small shapes gain from more, shorter ones
    while (kps > 16 && (long long)B * Hkv * ((capacity + kps - 1) / kps) < std::max(cus, 1)) kps /= 2;
    p.keys_per_split = kps;
    p.nsplit = std::max(1, (capacity + p.keys_per_split - 1) / p.keys_per_split);
    p.part_rows = (size_t)B * Hkv * p.nsplit * p.rows_padded;
    // one work-group per (split, sequence, KV head) on the grid's x extent
    if ((long long)p.nsplit * B * Hkv >= (1LL << 31)) p.ok = false;
  } else {
    // one wave per 16-row block, 1, 2 or 4 blocks per work-group.  Blocks
    // of 4 run as 8 waves in two key groups over a 128 KB ring, one work-
    // group per compute unit; smaller ones hold a 64 KB ring, two per unit
    // (stream_cfg).  The grid is that many work-groups, whatever the
    // lengths.
    p.row_blocks = blocks16 <= 1 ? 1 : (blocks16 == 2 ? 2 : 4);
    p.row_groups = (blocks16 + p.row_blocks - 1) / p.row_blocks;
    p.rows_wg = p.row_blocks * 16;
    p.rows_padded = p.row_groups * p.rows_wg;
    p.key_groups = stream_cfg(p.row_blocks).kg;
    const long long pairs = (long long)B * Hkv * p.row_groups;
    // at least 4 tiles per work-group when every sequence is at capacity
    const long long tiles_cap = pairs * ((capacity + kTile - 1) / kTile);
    p.stream_wgs = (int)std::max(1LL, std::min((long long)std::max(1, cus) * stream_cfg(p.row_blocks).per_cu,
                                               tiles_cap / 4));
    // tile indices are 32-bit on the device
    if (pairs * ((capacity + kTile - 1) / kTile) >= (1LL << 30)) p.ok = false;
    p.part_rows = (size_t)(pairs + p.stream_wgs) * p.key_groups * p.rows_wg;
  }
  p.workspace_bytes = p.part_rows * ((size_t)D + 1) * sizeof(float);
  return p;
}

hipError_t launch_verify(const VerifyArgs& a, const VerifyPlan& p, int dtype, hipStream_t st) {
  const bool paged = a.page_table != nullptr;
  hipError_t e;
  if (dtype == 0) {
    const size_t lds = (size_t)p.rows * p.keys_per_split * 8 + (size_t)p.rows * 16 +
                       (size_t)p.rows * (a.D + 1) * 4 + (size_t)2 * p.keys_per_split * (a.D + 1) * 4;
    dim3 grid((unsigned)((long long)p.nsplit * a.Hkv * a.B));
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
  if (dtype == 0)
    hipLaunchKernelGGL(verify_merge, dim3(a.Hkv * a.B, (p.rows + 3) / 4), dim3(256), 0, st, a,
                       p.keys_per_split, p.nsplit, p.rows_padded, paged ? 1 : 0);
  else
    hipLaunchKernelGGL(verify_stream_merge, dim3(a.B * a.Hkv * p.row_groups, (p.rows_wg + 3) / 4),
                       dim3(256), 0, st, a, p.stream_wgs, p.row_groups, p.key_groups, p.rows_wg,
                       paged ? 1 : 0);
  return hipGetLastError();
}

}  // namespace sd
