// Latent-guided visual-token compression (SpecFLASH Sec. 3.2, Eq. 3):
//   out[b][:, hs] = softmax(scale * Cq[:, hs] F_V[b][:, hs]^T) F_V[b][:, hs]
// for every head slice hs.  The query set Cq is shared by the batch and F_V
// is both key and value, so one staged tile of F_V feeds both products.
//
// bf16 path (matrix cores), grid (sequence x head x latent tile, token split):
//   - a work-group of NW waves owns NW * 32 latents of one (sequence, head);
//     each wave keeps its 32 latents' query fragments in registers;
//   - 64-token tiles of F_V[b][:, hs] are copied HBM -> LDS with the
//     global_load_lds DMA (no VGPR staging) into a 4-buffer ring, the 16-byte
//     pieces of each token XOR-swizzled so that every read pattern below is
//     free of LDS bank conflicts;
//   - each tile is converted bf16 -> fp16 once per work-group (exact for
//     zero and |F_V| in [2^-17, 65280], rounded to nearest otherwise, so
//     larger magnitudes become inf; a wave whose outputs then come out
//     non-finite, or all below 2^-12, recomputes its latents exactly in float64
//     (compress_exact_wave)), so that P V runs on fp16 matrix cores:
//     S^T = F_V Cq^T (lane = one latent row), online softmax in fp32 with
//     exp2, P (in [0, 2^15]) rounded to fp16, O^T += F_V^T P^T.  Eight-wave
//     groups over 128-channel heads take the scores from the bf16 tile as
//     copied (bf16 matrix cores) and convert into a second, channel-major
//     fp16 copy whose P V fragments are plain 16-byte reads; the others
//     convert in place and read F_V^T fragments by transposing reads;
//   - latent tiles of one (sequence, head) are placed on the same XCD
//     (work-groups are dealt to the 8 XCDs round-robin) so their F_V reads
//     hit the same L2.
// When the tokens are split across work-groups (small grids), each split
// writes a normalised partial (o, lse) and a merge kernel combines them.
//
// fp32 inputs, and bf16 inputs with 256-channel heads: a plain kernel
// (scores in LDS, float64 arithmetic) with the same partial format.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

constexpr int kTok = 64;   // tokens per LDS tile of the bf16 kernel
constexpr int kQ8MaxSplit = 16384;   // tokens per split of the int8 kernel (their exponents sit in LDS)

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;


// LDS swizzle of the F_V tile rows (see lds_swizzle)
template <int DH>
__device__ __forceinline__ constexpr int swz(int t) {
  return lds_swizzle<DH / 8>(t);
}

// Compile-time loop: f(std::integral_constant<int, I>{}) for I = B .. E-1.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Byte offset of a ring slot from the ring's start: a compile-time constant
// (CtOff, folded into the LDS instruction's offset field) or a runtime value
// added to the lane's base address.
template <int V>
using CtOff = std::integral_constant<int, V>;
template <int OFF, int V>
__device__ __forceinline__ u32x4 rd_b128(uint32_t base, CtOff<V>) { return lds_read_b128_off<OFF + V>(base); }
template <int OFF>
__device__ __forceinline__ u32x4 rd_b128(uint32_t base, uint32_t rt) { return lds_read_b128_off<OFF>(base + rt); }
template <int OFF, int V>
__device__ __forceinline__ u32x2 rd_tr16(uint32_t base, CtOff<V>) { return lds_read_tr16_b64_off<OFF + V>(base); }
template <int OFF>
__device__ __forceinline__ u32x2 rd_tr16(uint32_t base, uint32_t rt) { return lds_read_tr16_b64_off<OFF>(base + rt); }
template <int OFF, int V>
__device__ __forceinline__ void wr_b128(uint32_t base, CtOff<V>, const u32x4& v) { lds_write_b128_off<OFF + V>(base, v); }
template <int OFF>
__device__ __forceinline__ void wr_b128(uint32_t base, uint32_t rt, const u32x4& v) { lds_write_b128_off<OFF>(base + rt, v); }

// Map the linear work-group id to (sequence*head, latent tile) so that the
// latent tiles of one (sequence, head) land on the same XCD.
__device__ __forceinline__ void map_tile(int lin, int n_bh, int n_lt, int& bh, int& lt) {
  if ((n_bh & 7) == 0) {
    const int xcd = lin & 7, slot = lin >> 3;
    lt = slot % n_lt;
    bh = xcd + 8 * (slot / n_lt);
  } else {
    bh = lin / n_lt;
    lt = lin % n_lt;
  }
}

// One work-group = NW waves x 32 latents of one (sequence, head), one token
// split.  64-token tiles of F_V[b][:, hs] are copied HBM -> LDS by the
// global_load_lds DMA into a ring of four buffers.  One tile ahead of its
// score step, the work-group converts a tile from bf16 to fp16 (each
// 16-byte piece once per work-group), so every wave then runs the P V
// product on fp16 matrix cores with no per-wave conversion:
//   S^T = F_V Cq^T   (lane = one latent row, 16 tokens per tile and row)
//   O^T += F_V^T P^T (P = exp2(s - m) in [0, 2^15] rounded to fp16)
// Eight-wave groups with 128-channel heads (CM below) run the scores on the
// bf16 tile itself and write the fp16 tile channel-major into a second ring,
// so an F_V^T fragment is one 16-byte read; the other shapes convert in
// place, run the scores on fp16, and read F_V^T by the transposing
// ds_read_b64_tr_b16 (two reads per fragment).
// The loop is software-pipelined across tiles (scores of the next tile under
// the exponentials of the current one) and split into groups whose LDS
// reads are issued one group ahead.  The running maximum is raised (O, l
// rescaled) only when a row's scores exceed it by 2^15, which each lane
// checks on its own scores against a per-row threshold, and the token mask
// is applied only on the tail tile.  Tile reads and the in-place conversion
// are inline asm, and each step has one counted wait for its copies and
// one fence-free barrier (for eight-wave groups placed before the step's
// last group, so the next step's first reads overlap that group's work).
template <int NW, int DH, bool IN8>
constexpr bool kChannelMajor = !IN8 && NW == 8 && DH == 128;
template <int NW, int DH, bool IN8>
struct CompressLds {
  static constexpr bool CM = kChannelMajor<NW, DH, IN8>;
  unsigned char ring[4][64 * DH * 2];                       // bf16 tiles (CM) / fp16 tiles
  unsigned char tr[CM ? 4 : 1][CM ? 64 * DH * 2 : 16];      // CM: channel-major fp16 tiles
  unsigned char stage[IN8 ? 4 : 1][IN8 ? 64 * DH : 16];    // int8 staging tiles
  int8_t sexp[IN8 ? kQ8MaxSplit : 4];                      // int8: the split's token exponents
};

// The matrix-core pass of a work-group (NW waves x 32 latents of one
// (sequence, head), one token split).  Returns, per thread, the range flags
// of its outputs (bf16 input): bit 0 set when an accumulator is not finite,
// bit 1 set when some output it wrote has magnitude 2^-12 or more.
template <int NW, int DH, bool IN8>
__device__ __forceinline__ unsigned compress_pass(const CompressArgs a, int n_bh, int n_lt, int tokens_per_split,
                                                  int nsplit, CompressLds<NW, DH, IN8>& sm) {
  constexpr int TT = 64;                    // tokens per tile
  constexpr int DC = DH / 32;               // 32-channel slices (QK)
  constexpr int DB = DH / 16;               // 16-channel output blocks (PV)
  constexpr int PK = DH / 8;                // 16-byte fp16 pieces per token
  constexpr int ROW = DH * 2;               // fp16 bytes per token row
  constexpr int TILE_BYTES = TT * ROW;
  constexpr int IN_ROW = IN8 ? DH : DH * 2; // input bytes per token row
  constexpr int IN_PK = IN_ROW / 16;        // 16-byte input pieces per token
  constexpr int IN_PIECES = TT * IN_PK;     // per tile
  constexpr int DMA = IN_PIECES / 64;       // 64-lane copies per tile
  constexpr int DMA_PER_WAVE = DMA / NW;
  constexpr int CVT_PER_THREAD = IN_PIECES / (NW * 64);   // input pieces converted per thread
  constexpr int NBUF = 4;
  constexpr float kRescale = 15.f;      // P = exp2(s - m) <= 2^15 < the fp16 maximum
  static_assert(DMA % NW == 0 && IN_PIECES % (NW * 64) == 0, "tile work must split evenly");
  static_assert(!IN8 || DH == 128, "int8 input: 128-channel heads");
  // CM (eight-wave groups, 128-channel heads, bf16 input): the scores read
  // the bf16 tile as copied, on bf16 matrix cores; the conversion writes an
  // fp16 copy of the tile in channel-major order, from which the P V
  // fragments are plain 16-byte reads.  Otherwise the tile is converted in
  // place and the P V fragments come from transposing reads.
  constexpr bool CM = kChannelMajor<NW, DH, IN8>;
  // fp16 tiles (bf16 input: the copy lands here and is converted in place;
  // int8 input: converted here from the staging ring)
  auto& ring = sm.ring;
  auto& stage = sm.stage;
  auto& sexp = sm.sexp;
  static_assert(sizeof(sm.ring[0]) == TILE_BYTES, "ring slot size");
  static_assert(!CM || (CVT_PER_THREAD == 2 && sizeof(sm.tr[0]) == TILE_BYTES), "channel-major copy: two pieces per thread");

  int bh, lt;
  map_tile(blockIdx.x, n_bh, n_lt, bh, lt);
  const int split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tok0 = split * tokens_per_split;
  const int tok1 = min(a.N, tok0 + tokens_per_split);
  const int tid = threadIdx.x;
  // the wave index in a scalar register, so that the copies' LDS
  // destinations (M0) are formed by scalar arithmetic
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, G = lane >> 4, c = lane & 15;
  const int lat0 = lt * NW * 32 + w * 32;

  // query fragments (B operand): lane holds Cq[lat0 + rb*16 + c][h*DH + dc*32 + 8G ..],
  // bf16 as stored when the scores read the bf16 tile (CM), else fp16
  Pack8 qf[2][DC];
  if constexpr (IN8) {
    const int8_t* lat = static_cast<const int8_t*>(a.latents);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int r = lat0 + rb * 16 + c;
      const int e = r < a.C ? min(max((int)a.latent_exp[r], -14), 9) : 0;
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        const u32x2 q = r < a.C ? *reinterpret_cast<const u32x2*>(lat + (size_t)r * a.d + h * DH + dc * 32 + 8 * G)
                                : u32x2{0u, 0u};
        u32x4 lo, hi;
        i8x16_to_f16_pow2(u32x4{q[0], q[1], 0u, 0u}, e, lo, hi);
        qf[rb][dc].u = lo;
      }
    }
  } else {
    const uint16_t* lat = static_cast<const uint16_t*>(a.latents);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int r = lat0 + rb * 16 + c;
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = r < a.C ? *reinterpret_cast<const u32x4*>(lat + (size_t)r * a.d + h * DH + dc * 32 + 8 * G)
                       : u32x4{0u, 0u, 0u, 0u};
        if constexpr (!CM) {
#pragma unroll
          for (int e = 0; e < 4; ++e) pk.u[e] = bf16x2_to_f16x2(pk.u[e]);
        }
        qf[rb][dc] = pk;
      }
    }
  }

  // o[rb][0..DB-1]: O^T blocks; o[rb][DB]: the row sums l, formed on the
  // matrix cores from the same fp16 P (a "ones" row as the A fragment puts
  // l of latent c at accumulator row 0, i.e. lane c of group 0, element 0)
  float m[2] = {-INFINITY, -INFINITY};
  floatx4 o[2][DB + 1];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int db = 0; db <= DB; ++db) o[rb][db] = floatx4{0.f, 0.f, 0.f, 0.f};
  f16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (_Float16)(c == 0 ? 1.f : 0.f);

  const unsigned char* fbase = static_cast<const unsigned char*>(a.feats) +
                              ((size_t)b * a.N * a.d + h * DH) * (IN8 ? 1 : 2);
  const int ntiles = (tok1 - tok0 + TT - 1) / TT;
  const int last = ntiles - 1;
  if constexpr (IN8) {
    // the split's token exponents, once, before any copy is in flight
    const int8_t* fe = a.feat_exp + (size_t)b * a.N + tok0;
    for (int i = tid; i < tok1 - tok0; i += NW * 64) sexp[i] = fe[i];
  }

  // copy i of this wave moves input pieces P = (w * DMA_PER_WAVE + i) * 64 +
  // lane: token P / IN_PK.  bf16: LDS slot P % PK holds global piece
  // slot ^ swizzle(token) of the fp16 tile; int8: the staging tile is plain
  // token-major.  Tokens past the split re-read its last token.  The
  // address is the tile's first row (uniform, scalar registers) plus a
  // 32-bit lane offset formed with a 24-bit multiply-add (token < 64, row
  // stride < 2^23), so the copy needs two full-rate vector ops.
  const uint32_t row_bytes = (uint32_t)a.d * (IN8 ? 1u : 2u);
  auto issue = [&](int tile, int slot) {
    const int t0 = tok0 + tile * TT;
    const int lim = tok1 - 1 - t0;            // last token of the split, tile-relative (>= 0)
    const unsigned char* tbase = fbase + (size_t)t0 * row_bytes;
    unsigned char* buf = IN8 ? stage[slot] : ring[slot];
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const int P = (w * DMA_PER_WAVE + i) * 64 + lane;
      const int tk = P / IN_PK, piece = P % IN_PK;
      const int src_piece = IN8 ? piece : (piece ^ swz<DH>(tk));
      const uint32_t off = __umul24((uint32_t)min(tk, lim), row_bytes) + (uint32_t)src_piece * 16u;
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)(tbase + off),
                                       (lds_void*)(buf + (w * DMA_PER_WAVE + i) * 1024), 16, 0, 0);
    }
  };
  // int8 input: input piece i of this thread (token tk, channels 16 p8 ..)
  // becomes fp16 pieces 2 p8 and 2 p8 + 1 of token tk (swizzled slots),
  // written as soon as they are formed (the fp16 slot is not read before
  // the next step's barrier)
  auto piece_token = [&](int i) { return (i * NW * 64 + tid) / IN_PK; };
  auto write_f16 = [&](uint32_t base, int i, const u32x4& lo, const u32x4& hi) {
    const int tk = piece_token(i), p8 = (i * NW * 64 + tid) % IN_PK;
    lds_write_b128(base + tk * ROW + (((2 * p8) ^ swz<DH>(tk)) * 16), lo);
    lds_write_b128(base + tk * ROW + (((2 * p8 + 1) ^ swz<DH>(tk)) * 16), hi);
  };
  // LDS address of the exponent of input piece i of tile `tile` (the tile
  // clamped as the copies are, the token clamped to the split)
  const uint32_t sexp_base = lds_addr(sexp);
  auto exp_addr = [&](int tile, int i) {
    return sexp_base + (uint32_t)min(min(tile, last) * TT + piece_token(i), tok1 - tok0 - 1);
  };
  // Channel-major fp16 copy (CM), laid out by its fragments: a slot holds
  // the 16-byte piece (hf, db, G, c) at byte hf * 8192 + db * 1024 +
  // G * 256 + c * 16, namely channel 16 db + c at tokens 32 hf + 4 G +
  // {0..3} and 32 hf + 16 + 4 G + {0..3} (the K order of the P V products).
  // The P V fragment of lane (c, G) for half hf and value block db is then
  // the piece at its own lane offset, and the conversion, in which wave w
  // takes value block w and thread (G, c) the pieces (hf, w, G, c) of both
  // halves, writes at its thread offset: both are 1024 contiguous bytes per
  // wave and instruction, free of bank conflicts.  Each piece is two
  // transposing reads of 4 tokens x 16 channels of the bf16 tile (tokens
  // 32 hf + 16 blk + 4 G + {0..3}, lane c receiving channel 16 w + c), the
  // pattern of the in-place kernel's F_V^T reads.
  uint32_t cm_rd = 0u, cm_wr = 0u;
  if constexpr (CM) {
    const int trow = 4 * G + (c >> 2);                         // token row of half 0, block 0
    cm_rd = lds_addr(ring[0]) + trow * ROW + (((2 * w + ((c & 3) >> 1)) ^ swz<DH>(trow)) * 16) + (c & 1) * 8;
    cm_wr = lds_addr(sm.tr[0]) + tid * 16;
  }
  // conversion of this thread's pieces of a tile: bf16 in place (or, CM,
  // into the channel-major copy), or int8 from the staging slot into the
  // fp16 slot
  auto convert = [&](int slot, int tile) {
    const uint32_t base = lds_addr(ring[slot]);
    if constexpr (CM) {
      const uint32_t rs = (uint32_t)slot * TILE_BYTES;
      u32x4 v[2];
      static_for<0, 2>([&](auto jtag) {
        constexpr int j = decltype(jtag)::value;
        const u32x2 r0 = lds_read_tr16_b64_off<j * 32 * ROW>(cm_rd + rs);
        const u32x2 r1 = lds_read_tr16_b64_off<j * 32 * ROW + 16 * ROW>(cm_rd + rs);
        v[j] = u32x4{r0[0], r0[1], r1[0], r1[1]};
      });
      lds_wait();
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        tie(v[j]);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[j][e] = bf16x2_to_f16x2(v[j][e]);
        lds_write_b128(cm_wr + rs + j * 8192, v[j]);
      }
    } else if constexpr (IN8) {
      const uint32_t sbase = lds_addr(stage[slot]);
      u32x4 v[CVT_PER_THREAD];
      int e[CVT_PER_THREAD];
#pragma unroll
      for (int i = 0; i < CVT_PER_THREAD; ++i) {
        v[i] = lds_read_b128(sbase + (i * NW * 64 + tid) * 16);
        e[i] = lds_read_i8(exp_addr(tile, i));
      }
      lds_wait();
#pragma unroll
      for (int i = 0; i < CVT_PER_THREAD; ++i) {
        tie(v[i]);
        tie(e[i]);
        u32x4 lo, hi;
        i8x16_to_f16_pow2(v[i], min(max(e[i], -14), 9), lo, hi);
        write_f16(base, i, lo, hi);
      }
    } else {
      u32x4 v[CVT_PER_THREAD];
#pragma unroll
      for (int i = 0; i < CVT_PER_THREAD; ++i) v[i] = lds_read_b128(base + (i * NW * 64 + tid) * 16);
      lds_wait();
#pragma unroll
      for (int i = 0; i < CVT_PER_THREAD; ++i) {
        tie(v[i]);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[i][e] = bf16x2_to_f16x2(v[i][e]);
        lds_write_b128(base + (i * NW * 64 + tid) * 16, v[i]);
      }
    }
  };

  // Per-lane LDS bases (the tile offsets below are multiples of 16 tokens, so
  // token & 15 and the swizzle are fixed per lane).  Score fragments: token
  // kb*16 + c, piece dc*4 + G, one base per dc plus the immediate kb*16*ROW.
  // Transposed value reads: lane j of group G addresses token 4G + j/4 of a
  // 16-token block at channels db*16 + 4*(j%4), i.e. piece 2*db + ((j&3)>>1)
  // at byte 8*(j&1); one base per db plus the block's immediate offset.
  // The bases include the ring's start, so a slot is an offset from them.
  const uint32_t ring0 = lds_addr(ring[0]);
  uint32_t xbase[DC];
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) xbase[dc] = ring0 + c * ROW + ((dc * 4 + G) ^ swz<DH>(c)) * 16;
  uint32_t vbase[DB];
  {
    const int tt = 4 * G + (c >> 2);
#pragma unroll
    for (int db = 0; db < DB; ++db)
      vbase[db] = ring0 + tt * ROW + ((2 * db + ((c & 3) >> 1)) ^ swz<DH>(tt)) * 16 + (c & 1) * 8;
  }
  // CM: P V fragments at the lane's offset in the channel-major copy; the
  // half and the value block are immediate offsets
  const uint32_t cm_v = CM ? lds_addr(sm.tr[0]) + lane * 16 : 0u;
  // this thread's conversion pieces: base of its input (ring or staging)
  constexpr int IN_TILE = IN8 ? TT * DH : TILE_BYTES;    // input slot bytes
  const uint32_t cvt_base = (IN8 ? lds_addr(stage[0]) : ring0) + tid * 16;

  // A negative scale is folded into the queries (softmax(s * q . x) =
  // softmax(|s| * (-q) . x)), so the loop below only handles sl2 >= 0.
  float sl2 = a.scale_log2;
  if (sl2 < 0.f) {
    sl2 = -sl2;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc)
#pragma unroll
        for (int e = 0; e < 4; ++e) qf[rb][dc].u[e] ^= 0x80008000u;
  }

  // one score product: bf16 tile and queries (CM) or fp16 ones
  auto qk_mfma = [](const u32x4& x, const Pack8& q, const floatx4& acc) {
    Pack8 pk;
    pk.u = x;
    if constexpr (CM)
      return mfma_bf16(pk.b, q.b, acc);
    else
      return mfma_f16(pk.h, q.h, acc);
  };
  // Scores of one 16-token block of a tile (4 reads, 2 * DC matrix-core ops):
  // s[rb] lane holds S[row rb*16 + c][token kb*16 + 4G + i].
#define SD_QK_READ(XR, SB, KB)                                                             \
  _Pragma("unroll") for (int dc = 0; dc < DC; ++dc)                                        \
    XR[dc] = lds_read_b128_off<(KB) * 16 * ROW>((SB) + xbase[dc]);
#define SD_QK_MFMA(XR, S, KB)                                                              \
  _Pragma("unroll") for (int rb = 0; rb < 2; ++rb) {                                       \
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};                                                    \
    _Pragma("unroll") for (int dc = 0; dc < DC; ++dc) acc = qk_mfma(XR[dc], qf[rb][dc], acc); \
    S[KB][rb] = acc;                                                                       \
  }

  // Row maxima of a tile's scores (in log2 units), and the raise of the
  // running maxima with the (rare) rescale of O and l.
  auto tile_max = [&](const floatx4 (&s)[4][2], float (&tmax)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float ext = s[0][rb][0];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) ext = fmaxf(ext, s[kb][rb][i]);
      // every tile holds a valid token, so the maximum is finite
      tmax[rb] = wave_max_across_groups(ext * sl2);
    }
  };
  auto raise_max = [&](const float (&tmax)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      if (__ballot(tmax[rb] > m[rb] + kRescale) != 0ull) {
        const float mnew = fmaxf(m[rb], tmax[rb]);
        const float alpha = fast_exp2(m[rb] - mnew);
#pragma unroll
        for (int db = 0; db <= DB; ++db) o[rb][db] *= alpha;
        m[rb] = mnew;
      }
    }
  };
  // Steady-state check of a tile: each lane compares the 16 scores it holds
  // of each row block with the row's threshold thr = (m + kRescale) / sl2 in
  // score units (+inf for sl2 = 0), without the cross-lane maxima, and keeps
  // its own maxima (lmax); only when some lane exceeds the threshold does the
  // step reduce lmax across the lanes and raise m.  A threshold off by an ulp
  // only lets P reach 2^15 (1 + 2^-23), still far inside the fp16 range.
  float thr[2], lmax[2];
  const float inv_sl2 = sl2 > 0.f ? 1.f / sl2 : 0.f;
  auto set_thresholds = [&]() {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) thr[rb] = sl2 > 0.f ? (m[rb] + kRescale) * inv_sl2 : INFINITY;
  };
  auto tile_exceeds = [&](const floatx4 (&s)[4][2]) {
    bool hit = false;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float ext = s[0][rb][0];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) ext = fmaxf(ext, s[kb][rb][i]);
      lmax[rb] = ext;
      hit = hit || ext > thr[rb];
    }
    return hit;
  };
  // tokens at or past the end of the split get score -inf (last tile only)
  auto mask_tail = [&](floatx4 (&s)[4][2], int t0) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (t0 + kb * 16 + 4 * G + i >= tok1) {
          s[kb][0][i] = -INFINITY;
          s[kb][1][i] = -INFINITY;
        }
  };
  // p = exp2(s * sl2 - m) in fp16, for one row block
#define SD_P_ROW(S, PF, RB)                                                                \
  {                                                                                        \
    const float nm = -m[RB];                                                               \
    _Pragma("unroll") for (int kb = 0; kb < 4; ++kb)                                       \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                                        \
        PF[kb >> 1][RB][(kb & 1) * 4 + i] = (_Float16)fast_exp2(fmaf(S[kb][RB][i], sl2, nm)); \
  }

  // O^T += F_V^T P^T for one 32-token half; the product's K index runs over
  // tokens {4G..4G+3, 16+4G..16+4G+3} of the half, the order of pf.
#define SD_PV_READ(VR, SB, HF)                                                             \
  _Pragma("unroll") for (int db = 0; db < DB; ++db) {                                      \
    VR[db][0] = lds_read_tr16_b64_off<(HF) * 32 * ROW>((SB) + vbase[db]);                  \
    VR[db][1] = lds_read_tr16_b64_off<(HF) * 32 * ROW + 16 * ROW>((SB) + vbase[db]);       \
  }
#define SD_PV_MFMA(VR, PF, HF)                                                             \
  {                                                                                        \
    _Pragma("unroll") for (int db = 0; db < DB; ++db) {                                    \
      Pack8 vv;                                                                            \
      vv.u = u32x4{VR[db][0][0], VR[db][0][1], VR[db][1][0], VR[db][1][1]};                \
      _Pragma("unroll") for (int rb = 0; rb < 2; ++rb)                                     \
        o[rb][db] = mfma_f16(vv.h, PF[HF][rb], o[rb][db]);                                 \
    }                                                                                      \
    _Pragma("unroll") for (int rb = 0; rb < 2; ++rb)                                       \
      o[rb][DB] = mfma_f16(ones, PF[HF][rb], o[rb][DB]);                                   \
  }
  // interleave: one matrix-core op, then N VALU ops, `cnt` times (one
  // scheduling pipeline per phase, named by ID)
#define SD_INTERLEAVE(cnt, N, ID)                                                          \
  _Pragma("unroll") for (int q_ = 0; q_ < (cnt); ++q_) {                                   \
    __builtin_amdgcn_sched_group_barrier(0x008, 1, ID);                                    \
    __builtin_amdgcn_sched_group_barrier(0x002, (N), ID);                                  \
  }

  // Ring schedule (4 buffers), software-pipelined across tiles.  Entering
  // step it, scur holds the scores of tile it and the running maxima already
  // cover them.  After one barrier the step runs NG groups; each waits for
  // its own LDS reads (issued one group earlier), issues the next group's
  // reads, then interleaves its matrix-core ops with VALU work:
  //   QK groups (one per 32-channel slice dc): scores of tile it+1,
  //     accumulated over dc (8 independent ops per group) | exponentials of
  //     tile it (one quarter of them per group for DH = 128)
  //   PV groups (4 value blocks of one half each): P V of tile it |
  //     conversion of tile it+2 (first half; in place, or CM into the
  //     channel-major slot of tile it+2, whose last reader, the P V of tile
  //     it-2, finished two barriers earlier), the lane-local threshold
  //     check of tile it+1 (second half)
  // and, when some lane's scores passed its threshold, takes the exact row
  // maxima and raises them (rare rescale) for the next step, while tile it+3
  // is in flight.  Every step issues one tile (re-reading the last past the
  // end) and converts one buffer (past the end one that is never read
  // again), so the wait counts are the same at every step and the groups
  // form one basic block.
  constexpr int NQK = DC;              // QK read groups
  constexpr int NPVH = DB / 4;         // PV read groups per half
  constexpr int NG = NQK + 2 * NPVH;
  constexpr int KPG = 4 / NQK;         // 16-token blocks per QK group
  issue(0, 0);
  issue(min(1, last), 1);
  issue(min(2, last), 2);
  wait_vm_then_barrier<2 * DMA_PER_WAVE>();           // tile 0 landed
  convert(0, 0);
  wait_vm_then_barrier<DMA_PER_WAVE>();               // tile 1 landed, tile 0 converted
  convert(1, 1);
  floatx4 scur[4][2];
  {
    const uint32_t sb = 0;                      // ring slot 0
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 xr[DC];
      if (kb == 0) SD_QK_READ(xr, sb, 0)
      if (kb == 1) SD_QK_READ(xr, sb, 1)
      if (kb == 2) SD_QK_READ(xr, sb, 2)
      if (kb == 3) SD_QK_READ(xr, sb, 3)
      lds_wait();
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) tie(xr[dc]);
      SD_QK_MFMA(xr, scur, kb)
    }
    if (last == 0) mask_tail(scur, tok0);
    float tmax[2];
    tile_max(scur, tmax);
    raise_max(tmax);
    set_thresholds();
  }

  // LDS reads of group g into the alternating register sets xr / vr (and
  // the conversion pieces cv with the first PV group)
  auto reads = [&](auto gtag, auto nb, auto vb, auto cb, u32x4 (&xr)[2][4],
                   u32x2 (&vr)[2][4][2], u32x4 (&cv)[CVT_PER_THREAD], int (&ce)[CVT_PER_THREAD], int etile,
                   auto tie_only) {
    constexpr int g = decltype(gtag)::value;
    constexpr bool T = decltype(tie_only)::value;
    if constexpr (g < NQK) {
      // fragment j = kk * DC + dc: 16-token block g * KPG + kk, channel
      // slice dc
      auto& x = xr[g & 1];
      if constexpr (T) {
#pragma unroll
        for (int j = 0; j < 4; ++j) tie(x[j]);
      } else {
        static_for<0, 4>([&](auto jtag) {
          constexpr int j = decltype(jtag)::value, kb = g * KPG + j / DC, dc = j % DC;
          x[j] = rd_b128<kb * 16 * ROW>(xbase[dc], nb);
        });
      }
    } else if constexpr (g < NG) {
      constexpr int q = g - NQK, hf = q / NPVH, pb = q % NPVH;
      auto& v = vr[g & 1];
      if constexpr (T) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          tie(v[d][0]);
          tie(v[d][1]);
        }
        if constexpr (q == 0) {
#pragma unroll
          for (int i = 0; i < CVT_PER_THREAD; ++i) {
            tie(cv[i]);
            if constexpr (IN8) tie(ce[i]);
          }
        }
      } else {
        if constexpr (CM) {
          static_for<0, 4>([&](auto dtag) {
            constexpr int d = decltype(dtag)::value;
            const u32x4 x = rd_b128<hf * 8192 + (4 * pb + d) * 1024>(cm_v, vb);
            v[d][0] = u32x2{x[0], x[1]};
            v[d][1] = u32x2{x[2], x[3]};
          });
        } else {
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            v[d][0] = rd_tr16<hf * 32 * ROW>(vbase[4 * pb + d], vb);
            v[d][1] = rd_tr16<hf * 32 * ROW + 16 * ROW>(vbase[4 * pb + d], vb);
          }
        }
        if constexpr (q == 0) {
          static_for<0, CVT_PER_THREAD>([&](auto itag) {
            constexpr int i = decltype(itag)::value;
            if constexpr (CM) {
              const u32x2 r0 = rd_tr16<i * 32 * ROW>(cm_rd, cb);
              const u32x2 r1 = rd_tr16<i * 32 * ROW + 16 * ROW>(cm_rd, cb);
              cv[i] = u32x4{r0[0], r0[1], r1[0], r1[1]};
            } else {
              cv[i] = rd_b128<i * NW * 64 * 16>(cvt_base, cb);
            }
            if constexpr (IN8) ce[i] = lds_read_i8(exp_addr(etile, i));
          });
        }
      }
    }
  };

  // LDS operations issued by reads() for group g
  constexpr auto reads_in = [](int g) {
    if (CM) return g < NQK ? 4 : (g < NG ? 4 + (g == NQK ? 2 * CVT_PER_THREAD : 0) : 0);
    return g < NQK ? 4 : (g < NG ? 8 + (g == NQK ? CVT_PER_THREAD * (IN8 ? 2 : 1) : 0) : 0);
  };

  // Eight-wave groups (DH = 128) move the step's barrier from its start to
  // the start of its last group: the conversion has been written back one
  // group earlier, so after that barrier the next step's first reads and
  // copy can be issued and overlap the last group's matrix-core work.
  // Smaller groups keep the barrier at the step start and wait for a
  // group's reads before issuing the next group's (they have no registers
  // to spare for both in flight).
  constexpr bool kRot = NW == 8 && NQK + NPVH < NG - 1;
  u32x4 xr[2][4];

  // one step; the mask flag (compile time) is set only for it = last - 1, so
  // the steady-state loop has no branch between its groups.  The ring phase
  // PH = it % NBUF is a compile-time constant in the unrolled main loop (the
  // slots' offsets then sit in the LDS instructions' offset fields) and -1
  // elsewhere (offsets added at run time).  Entering a step: tile it+1
  // converted by every wave, tile it+2 landed, the copy of tile it+3 issued
  // and (kRot) the first group's reads done.
  auto step = [&](int it, auto mask_tag, auto ph_tag) {
    constexpr int PH = decltype(ph_tag)::value;
    // offset of the slot of tile it + K in a ring of slots of SZ bytes
    auto slot = [&](auto k_tag, auto sz_tag) {
      constexpr int K = decltype(k_tag)::value, SZ = decltype(sz_tag)::value;
      if constexpr (PH >= 0)
        return CtOff<((PH + K) % NBUF) * SZ>{};
      else
        return (uint32_t)(((it + K) % NBUF) * SZ);
    };
    const auto nb = slot(CtOff<1>{}, CtOff<TILE_BYTES>{});        // scores of tile it+1
    const auto cs = slot(CtOff<2>{}, CtOff<TILE_BYTES>{});        // converted tile it+2
    const auto ci = slot(CtOff<2>{}, CtOff<IN_TILE>{});           // its input
    const auto vb = slot(CtOff<0>{}, CtOff<TILE_BYTES>{});        // P V of tile it
    const uint32_t cb = lds_addr(ring[(it + 2) % NBUF]);          // int8: converted tile, absolute
    u32x2 vr[2][4][2];
    u32x4 cv[CVT_PER_THREAD];
    int ce[CVT_PER_THREAD];
    floatx4 snext[4][2];
    f16x8 pf[2][2];
    bool exceed = false;
    if constexpr (!kRot) {
      // tile it+2 landed; tile it+1 converted by every wave; buffer it-1 free
      wait_vm_then_barrier<0>();
      reads(std::integral_constant<int, 0>{}, nb, vb, ci, xr, vr, cv, ce, it + 2, std::false_type{});
      issue(min(it + 3, last), (it + 3) % NBUF);
    }
    static_for<0, NG>([&](auto gtag) {
      constexpr int g = decltype(gtag)::value;
      // issue the next group's reads, then wait for this group's (the
      // next group's stay in flight)
      if constexpr (kRot) {
        reads(std::integral_constant<int, g + 1>{}, nb, vb, ci, xr, vr, cv, ce, it + 2, std::false_type{});
        lds_wait_n<reads_in(g + 1)>();
        reads(gtag, nb, vb, ci, xr, vr, cv, ce, it + 2, std::true_type{});
      } else {
        lds_wait();
        reads(gtag, nb, vb, ci, xr, vr, cv, ce, it + 2, std::true_type{});
        reads(std::integral_constant<int, g + 1>{}, nb, vb, ci, xr, vr, cv, ce, it + 2, std::false_type{});
      }
      if constexpr (kRot && g == NG - 1) {
        // tile it+2 converted by every wave, tile it+3 landed, buffer it
        // read by every wave: start the next step's first group and copy
        // tile it+4 into buffer it, under this group's matrix-core work
        wait_vm_then_barrier<0>();
        if constexpr (!decltype(mask_tag)::value) {
          reads(std::integral_constant<int, 0>{}, cs, vb, ci, xr, vr, cv, ce, it + 2, std::false_type{});
          issue(min(it + 4, last), it % NBUF);
        }
      }
      if constexpr (g == NQK + NPVH) {
        // conversion finished in the first half: write it back
        if constexpr (CM) {
          static_for<0, CVT_PER_THREAD>([&](auto itag) {
            constexpr int i = decltype(itag)::value;
            wr_b128<i * 8192>(cm_wr, cs, cv[i]);
          });
        } else if constexpr (!IN8) {
          static_for<0, CVT_PER_THREAD>([&](auto itag) {
            constexpr int i = decltype(itag)::value;
            wr_b128<i * NW * 64 * 16>(cvt_base, cs, cv[i]);
          });
        }
      }
      if constexpr (g < NQK) {
        // scores of tile it+1 for the 16-token blocks kb of this group, each
        // summed over the channel slices (2 KPG chains of DC dependent ops):
        // the blocks of tile it+1 come to life as those of tile it die, so
        // the two tiles' scores hold about 40 registers rather than 64
        const auto& x = xr[g & 1];
#pragma unroll
        for (int kk = 0; kk < KPG; ++kk) {
          const int kb = g * KPG + kk;
#pragma unroll
          for (int dc = 0; dc < DC; ++dc) {
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
              snext[kb][rb] = qk_mfma(x[kk * DC + dc], qf[rb][dc], dc == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : snext[kb][rb]);
          }
        }
        // exponentials of the same blocks of tile it: pf[kb / 2][rb]
#pragma unroll
        for (int kk = 0; kk < KPG; ++kk) {
          const int kb = g * KPG + kk;
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) {
            const float nm = -m[rb];
#pragma unroll
            for (int i = 0; i < 4; ++i)
              pf[kb >> 1][rb][(kb & 1) * 4 + i] = (_Float16)fast_exp2(fmaf(scur[kb][rb][i], sl2, nm));
          }
        }
        SD_INTERLEAVE(8, 2, g + 1)
      } else {
        constexpr int q = g - NQK, hf = q / NPVH, pb = q % NPVH;
        if constexpr (q == 0 && decltype(mask_tag)::value) mask_tail(snext, tok0 + last * TT);
        const auto& v = vr[g & 1];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          Pack8 vv;
          vv.u = u32x4{v[d][0][0], v[d][0][1], v[d][1][0], v[d][1][1]};
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) o[rb][4 * pb + d] = mfma_f16(vv.h, pf[hf][rb], o[rb][4 * pb + d]);
        }
        if constexpr (pb == NPVH - 1) {
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) o[rb][DB] = mfma_f16(ones, pf[hf][rb], o[rb][DB]);
        }
        if constexpr (hf == 0) {
          // conversion of tile it+2, spread over the first half
#pragma unroll
          for (int i = pb; i < CVT_PER_THREAD; i += NPVH) {
            if constexpr (IN8) {
              u32x4 lo, hi;
              i8x16_to_f16_pow2(cv[i], min(max(ce[i], -14), 9), lo, hi);
              write_f16(cb, i, lo, hi);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) cv[i][e] = bf16x2_to_f16x2(cv[i][e]);
            }
          }
        } else if constexpr (pb == NPVH - 1) {
          exceed = tile_exceeds(snext);
        }
        SD_INTERLEAVE(8 + (pb == NPVH - 1 ? 2 : 0), 2, g + 1)
      }
      if constexpr (kRot && g == NG - 1 && !decltype(mask_tag)::value) {
        // the next step's first group is complete before the loop edge
        lds_wait();
        reads(std::integral_constant<int, 0>{}, nb, vb, ci, xr, vr, cv, ce, it + 2, std::true_type{});
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    if (__ballot(exceed) != 0ull) {            // rare: exact maxima, raise, new thresholds
      float tmax[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) tmax[rb] = wave_max_across_groups(lmax[rb] * sl2);
      raise_max(tmax);
      set_thresholds();
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) scur[kb][rb] = snext[kb][rb];
  };
  if (kRot && last >= 1) {
    // tile 1 converted by every wave, tile 2 landed: the first group of step
    // 0, and the copy of tile 3
    wait_vm_then_barrier<0>();
    u32x2 vr0[2][4][2];
    u32x4 cv0[CVT_PER_THREAD];
    int ce0[CVT_PER_THREAD];
    const auto nb0 = CtOff<TILE_BYTES>{};        // ring slot 1
    reads(std::integral_constant<int, 0>{}, nb0, nb0, nb0, xr, vr0, cv0, ce0, 0, std::false_type{});
    issue(min(3, last), 3 % NBUF);
    lds_wait();
    reads(std::integral_constant<int, 0>{}, nb0, nb0, nb0, xr, vr0, cv0, ce0, 0, std::true_type{});
  }
  int it = 0;
  for (; it + NBUF < last; it += NBUF) {
    step(it, std::false_type{}, CtOff<0>{});
    step(it + 1, std::false_type{}, CtOff<1>{});
    step(it + 2, std::false_type{}, CtOff<2>{});
    step(it + 3, std::false_type{}, CtOff<3>{});
  }
  for (; it + 1 < last; ++it) step(it, std::false_type{}, CtOff<-1>{});
  if (last >= 1) step(last - 1, std::true_type{}, CtOff<-1>{});
  {
    // last tile (masked and covered by the maxima): softmax and P V
    wait_vm_then_barrier<0>();
    const uint32_t vb = (last % NBUF) * TILE_BYTES;   // ring slot of the last tile
    f16x8 pf[2][2];
    SD_P_ROW(scur, pf, 0)
    SD_P_ROW(scur, pf, 1)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      u32x2 vr[DB][2];
      if constexpr (CM) {
        static_for<0, DB>([&](auto dtag) {
          constexpr int db = decltype(dtag)::value;
          const u32x4 x = lds_read_b128_off<db * 1024>(cm_v + vb + hf * 8192);
          vr[db][0] = u32x2{x[0], x[1]};
          vr[db][1] = u32x2{x[2], x[3]};
        });
      } else {
        if (hf == 0) SD_PV_READ(vr, vb, 0)
        if (hf == 1) SD_PV_READ(vr, vb, 1)
      }
      lds_wait();
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        tie(vr[db][0]);
        tie(vr[db][1]);
      }
      SD_PV_MFMA(vr, pf, hf)
    }
  }
#undef SD_QK_READ
#undef SD_QK_MFMA
#undef SD_P_ROW
#undef SD_PV_READ
#undef SD_PV_MFMA
#undef SD_INTERLEAVE
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // no copy in flight at exit

  // normalise and write (directly, or as a partial for the merge)
  unsigned flags = 0u;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float lt_ = __shfl(o[rb][DB][0], c, 64);   // l of row c sits in lane c
    const int r = lat0 + rb * 16 + c;
    if (r >= a.C) continue;
    const float inv = lt_ > 0.f ? 1.f / lt_ : 0.f;
    if constexpr (!IN8) {
      // range verdict: an input beyond fp16 became inf and made the scores
      // or sums non-finite; inputs all far below 2^-8 give tiny outputs
      float amax = 0.f;
      bool fin = __builtin_isfinite(lt_) && __builtin_isfinite(m[rb]);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = o[rb][db][e] * inv;
          fin = fin && __builtin_isfinite(x);
          amax = fmaxf(amax, fabsf(x));
        }
      flags |= (fin ? 0u : 1u) | (amax >= 0.000244140625f ? 2u : 0u);
    }
    float* dst;
    if (nsplit == 1) {
      dst = a.out + ((size_t)b * a.C + r) * a.d + h * DH;
    } else {
      const size_t pr = ((size_t)bh * nsplit + split) * a.C + r;
      dst = a.part_o + pr * DH;
      if (G == 0) a.part_lse[pr] = lt_ > 0.f ? m[rb] + log2f(lt_) : -INFINITY;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<floatx4*>(dst + db * 16 + 4 * G) = o[rb][db] * inv;
  }
  return flags;
}

// Exact fallback of one wave's 32 latents when its first-pass outputs left
// the range fp16 holds exactly (an accumulator not finite, or every output
// below 2^-12): the same outputs (or split partials) recomputed in float64
// from the bf16 values.  Registers and global memory only (no LDS, no
// barrier), so the other waves of the work-group, still streaming tiles
// through the ring, are neither disturbed nor held.  Per latent row, lanes
// take 64 tokens at a time for the scores (online softmax over the chunks)
// and then channels for P F_V.  Slow, and only run for such inputs.
template <int DH>
__device__ __forceinline__ void compress_exact_wave(const CompressArgs& a, int b, int h, int bh, int split,
                                                    int nsplit, int tok0, int tok1, int lat0) {
  constexpr int NC = DH / 64;                       // channels per lane
  const int lane = threadIdx.x & 63;
  const uint16_t* F = static_cast<const uint16_t*>(a.feats) + (size_t)b * a.N * a.d + h * DH;
  const double scale = (double)a.scale;
  // the first pass's stores to these outputs complete before any rewrite
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
  const int lat1 = min(a.C, lat0 + 32);
  for (int r = lat0; r < lat1; ++r) {
    const uint16_t* q = static_cast<const uint16_t*>(a.latents) + (size_t)r * a.d + h * DH;
    double m = -INFINITY, l = 0.0, acc[NC];
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) acc[cc] = 0.0;
    for (int t0 = tok0; t0 < tok1; t0 += 64) {
      const int t = t0 + lane;
      double s = -INFINITY;
      if (t < tok1) {
        const uint16_t* f = F + (size_t)t * a.d;
        double x = 0.0;
        for (int e = 0; e < DH; ++e) x = fma((double)bf16_bits_to_float(q[e]), (double)bf16_bits_to_float(f[e]), x);
        s = x * scale;
      }
      double mx = s;
      for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, 64));
      const double mnew = fmax(m, mx);               // finite: lane 0 holds a token
      const double p = t < tok1 ? exp(s - mnew) : 0.0;
      double sum = p;
      for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
      const double alpha = exp(m - mnew);            // 0 on the first chunk
      m = mnew;
      l = l * alpha + sum;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) acc[cc] *= alpha;
      const int nt = min(64, tok1 - t0);
      for (int j = 0; j < nt; ++j) {
        const double pj = __shfl(p, j, 64);
        const uint16_t* f = F + (size_t)(t0 + j) * a.d;
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) acc[cc] = fma(pj, (double)bf16_bits_to_float(f[lane + 64 * cc]), acc[cc]);
      }
    }
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const float v = (float)(acc[cc] / l);
      const int e = lane + 64 * cc;
      if (nsplit == 1) {
        a.out[((size_t)b * a.C + r) * a.d + h * DH + e] = v;
      } else {
        const size_t pr = ((size_t)bh * nsplit + split) * a.C + r;
        a.part_o[pr * DH + e] = v;
        if (e == 0) a.part_lse[pr] = (float)((m + log(l)) * 1.4426950408889634);
      }
    }
  }
}

template <int NW, int DH, bool IN8>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2))) void compress_bf16(CompressArgs a, int n_bh, int n_lt,
                                                         int tokens_per_split, int nsplit) {
  __shared__ __align__(16) CompressLds<NW, DH, IN8> sm;
  if constexpr (IN8) {
    compress_pass<NW, DH, true>(a, n_bh, n_lt, tokens_per_split, nsplit, sm);
  } else {
    const unsigned f = compress_pass<NW, DH, false>(a, n_bh, n_lt, tokens_per_split, nsplit, sm);
    // the wave's verdict (no barrier): rerun its latents exactly when some
    // accumulator is not finite, or when it has latents and every output
    // is below 2^-12
    int bh, lt;
    map_tile(blockIdx.x, n_bh, n_lt, bh, lt);
    const int lat0 = lt * NW * 32 + (threadIdx.x >> 6) * 32;
    const bool nonfinite = __ballot((f & 1u) != 0u) != 0ull;
    const bool sized = __ballot((f & 2u) != 0u) != 0ull;
    if (nonfinite || (lat0 < a.C && !sized)) {
      const int split = blockIdx.y;
      const int tok0 = split * tokens_per_split, tok1 = min(a.N, tok0 + tokens_per_split);
      compress_exact_wave<DH>(a, bh / a.H, bh % a.H, bh, split, nsplit, tok0, tok1, lat0);
    }
  }
}

// ------------------------------------------------- fp32 (and bf16, dh 256)
// fp32 inputs, and bf16 inputs with 256-channel heads: grid (8-latent
// block, token split, sequence x head) with short token splits, so the work
// spreads over many compute units.  Scores, softmax and P F_V run in float64
// (literal Eq. 3 scores reach |s| ~ 60 for unit-variance inputs, where fp32
// rounding of s would already cost ~1e-5 of relative accuracy in the
// weights).  The block's queries and the split's feature rows are staged in
// LDS as floats (bf16 widened exactly) with coalesced loads (rows padded by
// one float so that lanes reading one channel of consecutive rows hit
// distinct banks); the scores of the block live in LDS.  Splits and
// (sequence, head) pairs beyond the grid's y / z extent are taken in
// grid-stride loops.
constexpr int kF32Rows = 8;


template <typename T>
__global__ __launch_bounds__(256) void compress_lds(CompressArgs a, int dh, int tokens_per_split, int nsplit) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lb = blockIdx.x;
  const int r0 = lb * kF32Rows;
  const int nr = min(kF32Rows, a.C - r0);
  const int DS = dh + 1;
  double* ss = reinterpret_cast<double*>(smem);                // [8][tokens_per_split]
  double* st = ss + (size_t)kF32Rows * tokens_per_split;        // [8][2]
  float* qs = reinterpret_cast<float*>(st + 2 * kF32Rows);      // [8][dh + 1]
  float* fs = qs + (size_t)kF32Rows * DS;                        // [tokens_per_split][dh + 1]
  const T* lat = static_cast<const T*>(a.latents);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const double scale = (double)a.scale;
  for (int bh = blockIdx.z; bh < a.B * a.H; bh += gridDim.z) {
    const int b = bh / a.H, h = bh % a.H;
    const T* F = static_cast<const T*>(a.feats) + (size_t)b * a.N * a.d + h * dh;
    for (int split = blockIdx.y; split < nsplit; split += gridDim.y) {
      const int tok0 = split * tokens_per_split;
      const int nt = min(a.N, tok0 + tokens_per_split) - tok0;
      __syncthreads();                          // the previous item's LDS reads are done
      {
        float* const qd[1] = {qs};
        const T* const qsrc[1] = {lat};
        stage_rows<4, 1, 4>(qd, DS, qsrc, [&](int r) { return (size_t)(r0 + r) * a.d + h * dh; }, nr, dh);
        float* const fd[1] = {fs};
        const T* const fsrc[1] = {F};
        stage_rows<8, 1, 4>(fd, DS, fsrc, [&](int t) { return (size_t)(tok0 + t) * a.d; }, nt, dh);
      }
      __syncthreads();
      // thread i: latent i / nt, token i % nt (consecutive lanes, consecutive tokens)
      for (int i = tid; i < nt * nr; i += blockDim.x) {
        const int r = i / nt, t = i - r * nt;
        const float* xr = fs + t * DS;
        const float* qr = qs + r * DS;
        double acc = 0.0;
#pragma unroll 8
        for (int e = 0; e < dh; ++e) acc = fma((double)qr[e], (double)xr[e], acc);
        ss[(size_t)r * tokens_per_split + t] = acc * scale;
      }
      __syncthreads();
      for (int r = w; r < nr; r += blockDim.x / 64) {
        double mx = -INFINITY;
        for (int t = lane; t < nt; t += 64) mx = fmax(mx, ss[(size_t)r * tokens_per_split + t]);
        for (int off = 32; off > 0; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off, 64));
        double sum = 0.0;
        for (int t = lane; t < nt; t += 64) {
          const double p = exp(ss[(size_t)r * tokens_per_split + t] - mx);
          ss[(size_t)r * tokens_per_split + t] = p;
          sum += p;
        }
        for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
        if (lane == 0) {
          st[2 * r] = mx;
          st[2 * r + 1] = sum;
        }
      }
      __syncthreads();
      for (int i = tid; i < nr * dh; i += blockDim.x) {
        const int r = i / dh, e = i - r * dh;
        const double* pr = ss + (size_t)r * tokens_per_split;
        double acc = 0.0;
#pragma unroll 8
        for (int t = 0; t < nt; ++t) acc = fma(pr[t], (double)fs[t * DS + e], acc);
        const double sum = st[2 * r + 1];
        const float v = (float)(acc / sum);
        if (nsplit == 1) {
          a.out[((size_t)b * a.C + r0 + r) * a.d + h * dh + e] = v;
        } else {
          const size_t pr_ = ((size_t)bh * nsplit + split) * a.C + r0 + r;
          a.part_o[pr_ * dh + e] = v;
          if (e == 0) a.part_lse[pr_] = (float)((st[2 * r] + log(sum)) * 1.4426950408889634);
        }
      }
    }
  }
}

// Combine token splits: one thread per (sequence x head, latent, 4
// channels).  Up to 16 splits are loaded at once; a running maximum
// rescales the sums between rounds as in the online softmax.  Acc is the
// accumulation type: float for the matrix-core path, double for the
// float64 path (whose many short splits would otherwise let fp32 rounding
// of the running sums grow past its tolerance).
constexpr int kMergeRound = 16;
template <typename Acc>
__global__ __launch_bounds__(256) void compress_merge(CompressArgs a, int dh, int nsplit) {
  const int d4n = dh / 4;
  const long long item = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long rows = (long long)a.B * a.H * a.C;
  if (item >= rows * d4n) return;
  const long long row = item / d4n;
  const int d4 = (int)(item - row * d4n);
  const int bh = (int)(row / a.C), r = (int)(row - (long long)bh * a.C);
  const int b = bh / a.H, h = bh - b * a.H;
  const float* lse = a.part_lse + (size_t)bh * nsplit * a.C + r;
  const float* po = a.part_o + ((size_t)bh * nsplit * a.C + r) * dh + d4 * 4;
  const size_t ostride = (size_t)a.C * dh;     // elements between splits
  Acc acc[4] = {0, 0, 0, 0};
  Acc mx = -INFINITY, wsum = 0;
  for (int s0 = 0; s0 < nsplit; s0 += kMergeRound) {
    float l[kMergeRound];
    floatx4 v[kMergeRound];
#pragma unroll
    for (int i = 0; i < kMergeRound; ++i) {
      const int s = s0 + i;
      l[i] = s < nsplit ? lse[(size_t)s * a.C] : -INFINITY;
      v[i] = s < nsplit ? *reinterpret_cast<const floatx4*>(po + s * ostride) : floatx4{0.f, 0.f, 0.f, 0.f};
    }
    float cm = l[0];
#pragma unroll
    for (int i = 1; i < kMergeRound; ++i) cm = fmaxf(cm, l[i]);
    const Acc nm = mx > (Acc)cm ? mx : (Acc)cm;
    if (nm == -INFINITY) continue;
    // weights from fp32 exponentials of the exactly formed differences (the
    // stored partial lse values are fp32, whose rounding is of the same
    // order); only the running sums need the wider type
    const Acc keep = mx == -INFINITY ? (Acc)0 : (Acc)exp2f((float)(mx - nm));
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] *= keep;
    wsum *= keep;
#pragma unroll
    for (int i = 0; i < kMergeRound; ++i) {
      const Acc wgt = l[i] == -INFINITY ? (Acc)0 : (Acc)exp2f((float)((Acc)l[i] - nm));
      wsum += wgt;
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += wgt * (Acc)v[i][e];
    }
    mx = nm;
  }
  const Acc inv = wsum > 0 ? (Acc)1 / wsum : (Acc)0;
  *reinterpret_cast<floatx4*>(a.out + ((size_t)b * a.C + r) * a.d + h * dh + d4 * 4) =
      floatx4{(float)(acc[0] * inv), (float)(acc[1] * inv), (float)(acc[2] * inv), (float)(acc[3] * inv)};
}

// Average pooling of the N tokens into C contiguous groups (the
// non-parametric compressor of the compression ablation, Sec. 4.3): group c
// holds tokens floor(c N / C) .. floor((c + 1) N / C) - 1, its feature is
// their mean.  Grid (channel blocks of 2048, C, B); each thread sums 8
// channels over the group's tokens in float64 (one 16-byte load per token
// for bf16 rows when aligned), so F_V is read once.
template <typename T>
__global__ __launch_bounds__(256) void avg_pool(const T* feats, float* out, int N, int C, int d) {
  const int c = blockIdx.y, b = blockIdx.z;
  const int lo = (int)((long long)c * N / C), hi = (int)((long long)(c + 1) * N / C);
  const int e0 = (blockIdx.x * 256 + threadIdx.x) * 8;
  if (e0 >= d) return;
  const T* src = feats + ((size_t)b * N + lo) * d + e0;
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const bool vec = sizeof(T) == 2 && e0 + 8 <= d && (d & 7) == 0 && (reinterpret_cast<uintptr_t>(feats) & 15) == 0;
  if (vec) {
#pragma unroll 4
    for (int t = lo; t < hi; ++t, src += d) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(src);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += (double)__uint_as_float(v[i] << 16);
        acc[2 * i + 1] += (double)__uint_as_float(v[i] & 0xffff0000u);
      }
    }
  } else {
    for (int t = lo; t < hi; ++t, src += d) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (e0 + i < d) {
          if constexpr (sizeof(T) == 2) {
            acc[i] += (double)bf16_bits_to_float(reinterpret_cast<const uint16_t*>(src)[i]);
          } else {
            acc[i] += (double)src[i];
          }
        }
      }
    }
  }
  const double inv = 1.0 / (double)(hi - lo);
  float* dst = out + ((size_t)b * C + c) * d + e0;
#pragma unroll
  for (int i = 0; i < 8; ++i)
    if (e0 + i < d) dst[i] = (float)(acc[i] * inv);
}

template <int NW, int DH, bool IN8>
hipError_t launch_bf16(const CompressArgs& a, const CompressPlan& p, hipStream_t st) {
  const int n_bh = a.B * a.H;
  dim3 grid(n_bh * p.lat_tiles, p.nsplit);
  hipLaunchKernelGGL((compress_bf16<NW, DH, IN8>), grid, dim3(NW * 64), 0, st, a, n_bh, p.lat_tiles,
                     p.tokens_per_split, p.nsplit);
  return hipGetLastError();
}

template <int DH, bool IN8>
hipError_t dispatch_nw(const CompressArgs& a, const CompressPlan& p, hipStream_t st) {
  switch (p.lat_tile / 32) {
    case 1: return launch_bf16<1, DH, IN8>(a, p, st);
    case 2: return launch_bf16<2, DH, IN8>(a, p, st);
    case 4: return launch_bf16<4, DH, IN8>(a, p, st);
    default: return launch_bf16<8, DH, IN8>(a, p, st);
  }
}

}  // namespace

CompressPlan plan_compress(int B, int N, int C, int d, int H, int dtype, int cus) {
  CompressPlan p{};
  p.dh = d / H;
  const long long n_bh = (long long)B * H;
  if (dtype == 0 || p.dh == 256) {
    p.lat_tile = kF32Rows;
    p.lat_tiles = (C + kF32Rows - 1) / kF32Rows;
    // short splits (64 tokens at most) so the grid spreads over the device;
    // the split's fp32 feature rows and the 8 queries (rows padded by one
    // float) and fp64 scores within 64 KB of LDS
    long long tps = 64;
    while (tps > 8 && (4LL * kF32Rows * (p.dh + 1) + 4LL * tps * (p.dh + 1) + 8LL * kF32Rows * tps +
                       16 * kF32Rows) > 65536)
      tps /= 2;
    // shorter splits (16 tokens at least) while the grid would leave
    // compute units idle (the float64 chains of a work-group are serial)
    while (tps > 16 && n_bh * p.lat_tiles * ((N + tps - 1) / tps) < std::max(cus, 1)) tps /= 2;
    p.tokens_per_split = (int)tps;
  } else {
    // 32 latents per wave; eight-wave groups (each F_V tile copied and
    // converted once for 256 latents) whenever there are more than 128
    int waves = C <= 32 ? 1 : (C <= 64 ? 2 : (C <= 128 ? 4 : 8));
    p.lat_tile = waves * 32;
    p.lat_tiles = (C + p.lat_tile - 1) / p.lat_tile;
    // split the tokens so that the grid fills the device in one round:
    // two work-groups per compute unit (one of eight waves, or with int8
    // input, whose staging ring doubles the LDS), keeping at least 128
    // tokens per split; int8 splits hold at most kQ8MaxSplit tokens
    const long long groups = n_bh * p.lat_tiles;
    const long long resident = (long long)std::max(cus, 1) * (waves == 8 || dtype == kCompressInt8 ? 1 : 2);
    long long nsplit = std::max(1LL, resident / groups);
    if (dtype == kCompressInt8) nsplit = std::max(nsplit, ((long long)N + kQ8MaxSplit - 1) / kQ8MaxSplit);
    long long tps = (N + nsplit - 1) / nsplit;
    tps = std::max(128LL, (tps + kTok - 1) / kTok * kTok);
    if (dtype == kCompressInt8) tps = std::min(tps, (long long)kQ8MaxSplit);
    p.tokens_per_split = (int)tps;
  }
  p.nsplit = std::max(1, (N + p.tokens_per_split - 1) / p.tokens_per_split);
  p.workspace_bytes = p.nsplit > 1
      ? (size_t)n_bh * p.nsplit * C * ((size_t)p.dh + 1) * sizeof(float) : 0;
  return p;
}

hipError_t launch_compress(const CompressArgs& a, const CompressPlan& p, int dtype, hipStream_t st) {
  hipError_t e;
  if (dtype == 0 || p.dh == 256) {
    const size_t lds = (size_t)kF32Rows * p.tokens_per_split * 8 + 16 * kF32Rows +
                       (size_t)kF32Rows * (p.dh + 1) * 4 + (size_t)p.tokens_per_split * (p.dh + 1) * 4;
    dim3 grid(p.lat_tiles, std::min(p.nsplit, 65535), std::min(a.B * a.H, 65535));
    if (dtype == 0)
      hipLaunchKernelGGL(compress_lds<float>, grid, dim3(256), lds, st, a, p.dh, p.tokens_per_split, p.nsplit);
    else
      hipLaunchKernelGGL(compress_lds<uint16_t>, grid, dim3(256), lds, st, a, p.dh, p.tokens_per_split,
                         p.nsplit);
    e = hipGetLastError();
  } else if (dtype == kCompressInt8) {
    e = dispatch_nw<128, true>(a, p, st);
  } else {
    e = p.dh == 128 ? dispatch_nw<128, false>(a, p, st) : dispatch_nw<64, false>(a, p, st);
  }
  if (e != hipSuccess || p.nsplit == 1) return e;
  const long long items = (long long)a.B * a.H * a.C * (p.dh / 4);
  const dim3 mgrid((unsigned)((items + 255) / 256));
  if (dtype == 0 || p.dh == 256)
    hipLaunchKernelGGL(compress_merge<double>, mgrid, dim3(256), 0, st, a, p.dh, p.nsplit);
  else
    hipLaunchKernelGGL(compress_merge<float>, mgrid, dim3(256), 0, st, a, p.dh, p.nsplit);
  return hipGetLastError();
}

hipError_t launch_avg_pool(const void* feats, float* out, int B, int N, int C, int d, int dtype, hipStream_t st) {
  const dim3 grid((d + 2047) / 2048, C, B);
  if (dtype == 0) {
    hipLaunchKernelGGL(avg_pool<float>, grid, dim3(256), 0, st, static_cast<const float*>(feats), out, N, C, d);
  } else {
    hipLaunchKernelGGL(avg_pool<uint16_t>, grid, dim3(256), 0, st, static_cast<const uint16_t*>(feats), out, N, C,
                       d);
  }
  return hipGetLastError();
}

}  // namespace sd
