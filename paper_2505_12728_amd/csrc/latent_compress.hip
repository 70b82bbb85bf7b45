// Latent-guided visual-token compression (SpecFLASH Sec. 3.2, Eq. 3):
//   out[b][:, hs] = softmax(scale * Cq[:, hs] F_V[b][:, hs]^T) F_V[b][:, hs]
// for every head slice hs.  The query set Cq is shared by the batch and F_V
// is both key and value, so one staged tile of F_V feeds both products.
//
// bf16 path (matrix cores), grid (sequence x head x latent tile, token split):
//   - a work-group of NW waves owns NW * 64 latents of one (sequence, head);
//     each wave keeps its 64 latents' query fragments in registers;
//   - 64-token tiles of F_V[b][:, hs] are copied HBM -> LDS with the
//     global_load_lds DMA (no VGPR staging), double-buffered, with the
//     16-byte pieces of each token XOR-swizzled by (token & 7) so that both
//     read patterns below spread over the LDS banks;
//   - S^T = F_V Cq^T on bf16 matrix cores (lane = one latent row), online
//     softmax in fp32 with exp2, then O^T += F_V^T P^T on fp16 matrix cores:
//     P (in [0, 1]) is rounded to fp16 and the F_V fragment read back with
//     the transposing ds_read_tr16_b64 is converted bf16 -> fp16, which is
//     exact for |F_V| in [2^-14, 65504];
//   - latent tiles of one (sequence, head) are placed on the same XCD
//     (work-groups are dealt to the 8 XCDs round-robin) so their F_V reads
//     hit the same L2.
// When the tokens are split across work-groups (small grids), each split
// writes a normalised partial (o, lse) and a merge kernel combines them.
//
// fp32 path: a plain kernel (scores in LDS, float64 arithmetic) with the
// same partial format, for fp32 inputs that need full fp32 accuracy.
#include <math.h>

#include <algorithm>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

constexpr int kTok = 64;   // tokens per LDS tile of the bf16 kernel

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;


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
// global_load_lds DMA into a ring of four buffers, so two tiles are in
// flight while a third is converted and a fourth computed.  One tile ahead
// of the compute, the work-group converts the tile in place from bf16 to
// fp16 (each 16-byte piece once per work-group), so every wave then runs
// both products on fp16 matrix cores with no per-wave conversion:
//   S^T = F_V Cq^T   (lane = one latent row, 16 tokens per tile and row)
//   O^T += F_V^T P^T (P = exp2(s - m) in [0, 256] rounded to fp16; F_V^T
//                     fragments via the transposing ds_read_b64_tr_b16)
// Token pieces are XOR-swizzled by (token & 7) in LDS.  The running maximum
// is raised (O, l rescaled) only when a row's scores exceed it by 2^8, and
// the token mask is applied only on the tail tile.  Tile reads and the
// in-place conversion are inline asm, and each step has one counted wait
// and one fence-free barrier.
template <int NW, int DH>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2))) void compress_bf16(CompressArgs a, int n_bh, int n_lt,
                                                         int tokens_per_split, int nsplit) {
  constexpr int TT = 64;                    // tokens per tile
  constexpr int DC = DH / 32;               // 32-channel slices (QK)
  constexpr int DB = DH / 16;               // 16-channel output blocks (PV)
  constexpr int PK = DH / 8;                // 16-byte pieces per token
  constexpr int ROW = DH * 2;               // bytes per token row
  constexpr int TILE_BYTES = TT * ROW;
  constexpr int DMA = TT * PK / 64;         // 64-lane copies per tile
  constexpr int DMA_PER_WAVE = DMA / NW;
  constexpr int CVT_PER_THREAD = TT * PK / (NW * 64);   // pieces converted per thread
  constexpr int NBUF = 4;
  constexpr float kRescale = 8.f;
  static_assert(DMA % NW == 0 && (TT * PK) % (NW * 64) == 0, "tile work must split evenly");
  __shared__ __align__(16) unsigned char ring[NBUF][TILE_BYTES];

  int bh, lt;
  map_tile(blockIdx.x, n_bh, n_lt, bh, lt);
  const int split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tok0 = split * tokens_per_split;
  const int tok1 = min(a.N, tok0 + tokens_per_split);
  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, G = lane >> 4, c = lane & 15;
  const int lat0 = lt * NW * 32 + w * 32;

  // query fragments (fp16, B operand): lane holds Cq[lat0 + rb*16 + c][h*DH + dc*32 + 8G ..]
  f16x8 qf[2][DC];
  {
    const uint16_t* lat = static_cast<const uint16_t*>(a.latents);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int r = lat0 + rb * 16 + c;
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = r < a.C ? *reinterpret_cast<const u32x4*>(lat + (size_t)r * a.d + h * DH + dc * 32 + 8 * G)
                       : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 4; ++e) pk.u[e] = bf16x2_to_f16x2(pk.u[e]);
        qf[rb][dc] = pk.h;
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

  const uint16_t* fbase = static_cast<const uint16_t*>(a.feats) + (size_t)b * a.N * a.d + h * DH;
  const int ntiles = (tok1 - tok0 + TT - 1) / TT;
  const int last = ntiles - 1;

  // copy i of this wave moves pieces P = (w * DMA_PER_WAVE + i) * 64 + lane:
  // token P / PK, LDS slot P % PK holding global piece slot ^ (token & 7)
  auto issue = [&](int tile, unsigned char* buf) {
    const int t0 = tok0 + tile * TT;
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const int P = (w * DMA_PER_WAVE + i) * 64 + lane;
      const int tk = P / PK, piece = P % PK;
      const int tg = min(t0 + tk, tok1 - 1);
      const uint16_t* src = fbase + (size_t)tg * a.d + ((piece ^ (tk & 7)) * 8);
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)src,
                                       (lds_void*)(buf + (w * DMA_PER_WAVE + i) * 1024), 16, 0, 0);
    }
  };
  // in-place bf16 -> fp16 conversion of this thread's pieces of a tile
  auto convert = [&](const unsigned char* buf) {
    const uint32_t base = lds_addr(buf);
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
  };

  // per-lane LDS offsets: score fragments (token kb*16 + c, channels
  // dc*32 + 8G ..) and transposed value reads (lane j of group G addresses
  // token 4G + j/4 (+16) of a 32-token half at channels db*16 + 4 (j%4))
  uint32_t xoff[4][DC];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      const int tk = kb * 16 + c;
      xoff[kb][dc] = tk * ROW + (((dc * 4 + G) ^ (tk & 7)) * 16);
    }
  auto voff = [&](int hf, int half16, int db) -> uint32_t {
    const int tk = hf * 32 + half16 * 16 + 4 * G + (c >> 2);
    const int ch = db * 16 + 4 * (c & 3);
    return tk * ROW + (((ch >> 3) ^ (tk & 7)) * 16) + (ch & 7) * 2;
  };

  const float sl2 = a.scale_log2;
  auto compute = [&](int it, const unsigned char* buf) {
    const uint32_t sb = lds_addr(buf);
    const int t0 = tok0 + it * TT;
    // S^T = F_V Cq^T for the tile: s[kb][rb] lane holds S[row rb*16 + c][token kb*16 + 4G + i]
    floatx4 s[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 xr[DC];
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) xr[dc] = lds_read_b128(sb + xoff[kb][dc]);
      lds_wait();
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) tie(xr[dc]);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dc = 0; dc < DC; ++dc) {
          Pack8 pk;
          pk.u = xr[dc];
          acc = mfma_f16(pk.h, qf[rb][dc], acc);
        }
        s[kb][rb] = acc;
      }
    }
    // Online softmax on raw scores: with sl2 = scale * log2(e), the row
    // maximum of s * sl2 is (max s) * sl2 for sl2 >= 0 and (min s) * sl2
    // otherwise, and p = exp2(s * sl2 - m) is one FMA and one exp.
    if (t0 + TT > tok1) {                   // tail tile: drop tokens past the split
      const float fill = sl2 >= 0.f ? -INFINITY : INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (t0 + kb * 16 + 4 * G + i >= tok1) {
            s[kb][0][i] = fill;
            s[kb][1][i] = fill;
          }
    }
    f16x8 pf[2][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float hi = s[0][rb][0], lo = s[0][rb][0];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          hi = fmaxf(hi, s[kb][rb][i]);
          lo = fminf(lo, s[kb][rb][i]);
        }
      // every tile holds a valid token, so the extreme is finite
      const float tmax = wave_max_across_groups((sl2 >= 0.f ? hi : lo) * sl2);
      if (__ballot(tmax > m[rb] + kRescale) != 0ull) {
        const float mnew = fmaxf(m[rb], tmax);
        const float alpha = fast_exp2(m[rb] - mnew);
#pragma unroll
        for (int db = 0; db <= DB; ++db) o[rb][db] *= alpha;
        m[rb] = mnew;
      }
      const float nm = -m[rb];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          pf[kb >> 1][rb][(kb & 1) * 4 + i] = (_Float16)fast_exp2(fmaf(s[kb][rb][i], sl2, nm));
    }
    // O^T += F_V^T P^T per 32-token half; the product's K index runs over
    // tokens {4G..4G+3, 16+4G..16+4G+3} of the half, the order of pf.
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      u32x2 vr[DB][2];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        vr[db][0] = lds_read_tr16_b64(sb + voff(hf, 0, db));
        vr[db][1] = lds_read_tr16_b64(sb + voff(hf, 1, db));
      }
      lds_wait();
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        tie(vr[db][0]);
        tie(vr[db][1]);
        Pack8 vv;
        vv.u = u32x4{vr[db][0][0], vr[db][0][1], vr[db][1][0], vr[db][1][1]};
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) o[rb][db] = mfma_f16(vv.h, pf[hf][rb], o[rb][db]);
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) o[rb][DB] = mfma_f16(ones, pf[hf][rb], o[rb][DB]);
    }
  };

  // Ring schedule: at step it, tile it (converted in step it-1) is computed,
  // tile it+1 (landed) is converted, tiles it+2 and it+3 are in flight.
  // Every step issues one tile (re-reading the last past the end), so the
  // wait count is the same at every step.
#pragma unroll
  for (int i = 0; i < NBUF - 1; ++i) issue(min(i, last), ring[i]);
  wait_vm_then_barrier<(NBUF - 2) * DMA_PER_WAVE>();   // tile 0 landed
  convert(ring[0]);
  for (int it = 0; it < ntiles; ++it) {
    // tile it+1 landed; tile it converted by every wave; slot it-1 free
    wait_vm_then_barrier<(NBUF - 3) * DMA_PER_WAVE>();
    issue(min(it + NBUF - 1, last), ring[(it + NBUF - 1) % NBUF]);
    if (it + 1 < ntiles) convert(ring[(it + 1) % NBUF]);
    compute(it, ring[it % NBUF]);
  }
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // no copy in flight at exit

  // normalise and write (directly, or as a partial for the merge)
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float lt_ = __shfl(o[rb][DB][0], c, 64);   // l of row c sits in lane c
    const int r = lat0 + rb * 16 + c;
    if (r >= a.C) continue;
    const float inv = lt_ > 0.f ? 1.f / lt_ : 0.f;
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
}

// ---------------------------------------------------------------- fp32
// fp32 inputs: grid (8-latent block, token split, sequence x head).  Scores,
// softmax and P F_V run in float64 (literal Eq. 3 scores reach |s| ~ 60 for
// unit-variance inputs, where fp32 rounding of s would already cost ~1e-5 of
// relative accuracy in the weights).  Scores of the block live in LDS.
constexpr int kF32Rows = 8;

__global__ __launch_bounds__(256) void compress_f32(CompressArgs a, int dh, int tokens_per_split,
                                                    int nsplit) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lb = blockIdx.x, split = blockIdx.y, bh = blockIdx.z;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = lb * kF32Rows;
  const int nr = min(kF32Rows, a.C - r0);
  const int tok0 = split * tokens_per_split;
  const int nt = min(a.N, tok0 + tokens_per_split) - tok0;
  if (nt <= 0) return;
  double* ss = reinterpret_cast<double*>(smem);                // [8][tokens_per_split]
  double* st = ss + (size_t)kF32Rows * tokens_per_split;        // [8][2]
  float* qs = reinterpret_cast<float*>(st + 2 * kF32Rows);      // [8][dh]
  const float* lat = static_cast<const float*>(a.latents);
  const float* F = static_cast<const float*>(a.feats) + (size_t)b * a.N * a.d + h * dh;
  const int tid = threadIdx.x;
  for (int i = tid; i < nr * dh; i += blockDim.x)
    qs[i] = lat[(size_t)(r0 + i / dh) * a.d + h * dh + i % dh];
  __syncthreads();
  const double scale = (double)a.scale;
  for (int i = tid; i < nt * nr; i += blockDim.x) {
    const int t = i / nr, r = i % nr;
    const float* xr = F + (size_t)(tok0 + t) * a.d;
    const float* qr = qs + r * dh;
    double acc = 0.0;
    for (int e = 0; e < dh; ++e) acc = fma((double)qr[e], (double)xr[e], acc);
    ss[(size_t)r * tokens_per_split + t] = acc * scale;
  }
  __syncthreads();
  const int w = tid >> 6, lane = tid & 63;
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
    const int r = i / dh, e = i % dh;
    double acc = 0.0;
    for (int t = 0; t < nt; ++t)
      acc = fma(ss[(size_t)r * tokens_per_split + t], (double)F[(size_t)(tok0 + t) * a.d + e], acc);
    const double sum = st[2 * r + 1];
    const float v = (float)(acc / sum);
    if (nsplit == 1) {
      a.out[((size_t)b * a.C + r0 + r) * a.d + h * dh + e] = v;
    } else {
      const size_t pr = ((size_t)bh * nsplit + split) * a.C + r0 + r;
      a.part_o[pr * dh + e] = v;
      if (e == 0) a.part_lse[pr] = (float)((st[2 * r] + log(sum)) * 1.4426950408889634);
    }
  }
}

// Combine token splits: grid (latent block of 64, sequence x head).
__global__ __launch_bounds__(256) void compress_merge(CompressArgs a, int dh, int nsplit) {
  const int bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = blockIdx.x * 64;
  const int d4n = dh / 4;
  const int nr = min(64, a.C - r0);
  for (int i = threadIdx.x; i < nr * d4n; i += blockDim.x) {
    const int r = r0 + i / d4n, d4 = i % d4n;
    float mx = -INFINITY;
    for (int s = 0; s < nsplit; ++s)
      mx = fmaxf(mx, a.part_lse[((size_t)bh * nsplit + s) * a.C + r]);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const size_t pr = ((size_t)bh * nsplit + s) * a.C + r;
      const float wgt = exp2f(a.part_lse[pr] - mx);
      wsum += wgt;
      acc += wgt * *reinterpret_cast<const floatx4*>(a.part_o + pr * dh + d4 * 4);
    }
    *reinterpret_cast<floatx4*>(a.out + ((size_t)b * a.C + r) * a.d + h * dh + d4 * 4) =
        acc * (1.f / wsum);
  }
}

template <int NW, int DH>
hipError_t launch_bf16(const CompressArgs& a, const CompressPlan& p, hipStream_t st) {
  const int n_bh = a.B * a.H;
  dim3 grid(n_bh * p.lat_tiles, p.nsplit);
  hipLaunchKernelGGL((compress_bf16<NW, DH>), grid, dim3(NW * 64), 0, st, a, n_bh, p.lat_tiles,
                     p.tokens_per_split, p.nsplit);
  return hipGetLastError();
}

template <int DH>
hipError_t dispatch_nw(const CompressArgs& a, const CompressPlan& p, hipStream_t st) {
  switch (p.lat_tile / 32) {
    case 1: return launch_bf16<1, DH>(a, p, st);
    case 2: return launch_bf16<2, DH>(a, p, st);
    default: return launch_bf16<4, DH>(a, p, st);
  }
}

}  // namespace

CompressPlan plan_compress(int B, int N, int C, int d, int H, int dtype) {
  CompressPlan p{};
  p.dh = d / H;
  const long long n_bh = (long long)B * H;
  if (dtype == 0) {
    p.lat_tile = kF32Rows;
    p.lat_tiles = (C + kF32Rows - 1) / kF32Rows;
    // fp64 scores of 8 latents + fp32 queries within 64 KB of LDS
    const long long cap = (65536 - 4LL * kF32Rows * p.dh - 16 * kF32Rows) / (8 * kF32Rows);
    p.tokens_per_split = (int)std::max(64LL, std::min(2048LL, cap / 64 * 64));
  } else {
    const int waves = C <= 32 ? 1 : (C <= 64 ? 2 : 4);   // 32 latents per wave
    p.lat_tile = waves * 32;
    p.lat_tiles = (C + p.lat_tile - 1) / p.lat_tile;
    // split the tokens until about 512 work-groups exist, keeping >= 256 tokens each
    const long long groups = n_bh * p.lat_tiles;
    long long nsplit = std::max(1LL, (512 + groups - 1) / groups);
    long long tps = (N + nsplit - 1) / nsplit;
    tps = std::max(256LL, (tps + kTok - 1) / kTok * kTok);
    p.tokens_per_split = (int)tps;
  }
  p.nsplit = std::max(1, (N + p.tokens_per_split - 1) / p.tokens_per_split);
  p.workspace_bytes = p.nsplit > 1
      ? (size_t)n_bh * p.nsplit * C * ((size_t)p.dh + 1) * sizeof(float) : 0;
  return p;
}

hipError_t launch_compress(const CompressArgs& a, const CompressPlan& p, int dtype, hipStream_t st) {
  hipError_t e;
  if (dtype == 0) {
    const size_t lds = (size_t)kF32Rows * p.tokens_per_split * 8 + 16 * kF32Rows +
                       (size_t)kF32Rows * p.dh * 4;
    dim3 grid(p.lat_tiles, p.nsplit, a.B * a.H);
    hipLaunchKernelGGL(compress_f32, grid, dim3(256), lds, st, a, p.dh, p.tokens_per_split,
                       p.nsplit);
    e = hipGetLastError();
  } else {
    e = p.dh == 128 ? dispatch_nw<128>(a, p, st) : dispatch_nw<64>(a, p, st);
  }
  if (e != hipSuccess || p.nsplit == 1) return e;
  hipLaunchKernelGGL(compress_merge, dim3((a.C + 63) / 64, a.B * a.H), dim3(256), 0, st, a, p.dh,
                     p.nsplit);
  return hipGetLastError();
}

}  // namespace sd
