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

constexpr int kTok = 64;   // tokens per LDS tile

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;

__device__ __forceinline__ int swz(int token) { return token & 7; }

__device__ __forceinline__ uint32_t cvt_bf16x2_to_f16x2(uint32_t v) {
  // two bf16 values -> two fp16 values (exact inside the fp16 range)
  const float lo = __uint_as_float(v << 16);
  const float hi = __uint_as_float(v & 0xffff0000u);
  auto h2 = __builtin_amdgcn_cvt_pkrtz(lo, hi);
  uint32_t r;
  __builtin_memcpy(&r, &h2, 4);
  return r;
}

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

template <int NW, int DH>
__global__ __launch_bounds__(NW * 64) void compress_bf16(CompressArgs a, int n_bh, int n_lt,
                                                         int tokens_per_split, int nsplit) {
  constexpr int DC = DH / 32;               // 32-channel slices (QK)
  constexpr int DB = DH / 16;               // 16-channel output blocks (PV)
  constexpr int PK = DH / 8;                // 16-byte pieces per token
  constexpr int TILE_BYTES = kTok * DH * 2;
  constexpr int LOADS = kTok * PK / 64;     // DMA instructions per tile
  constexpr int LOADS_PER_WAVE = LOADS / NW;
  static_assert(LOADS % NW == 0, "tile copy must split evenly over the waves");
  __shared__ __align__(16) unsigned char tile_buf[2][TILE_BYTES];

  int bh, lt;
  map_tile(blockIdx.x, n_bh, n_lt, bh, lt);
  const int split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tok0 = split * tokens_per_split;
  const int tok1 = min(a.N, tok0 + tokens_per_split);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, G = lane >> 4, c = lane & 15;
  const int lat0 = lt * NW * 64 + w * 64;

  // query fragments (B operand): lane holds Cq[lat0 + rb*16 + c][h*DH + dc*32 + 8G ..]
  bf16x8 qf[4][DC];
  const uint16_t* lat = static_cast<const uint16_t*>(a.latents);
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int r = lat0 + rb * 16 + c;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      Pack8 pk;
      pk.u = r < a.C ? *reinterpret_cast<const u32x4*>(lat + (size_t)r * a.d + h * DH + dc * 32 + 8 * G)
                     : u32x4{0u, 0u, 0u, 0u};
      qf[rb][dc] = pk.b;
    }
  }

  float m[4], l[4];
  floatx4 o[4][DB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  const uint16_t* fbase = static_cast<const uint16_t*>(a.feats) + (size_t)b * a.N * a.d + h * DH;
  const int ntiles = (tok1 - tok0 + kTok - 1) / kTok;

  // DMA one 64-token tile into buffer `buf`: instruction i of this wave moves
  // pieces P = (w * LOADS_PER_WAVE + i) * 64 + lane, LDS slot P, i.e. token
  // P / PK, slot P % PK, holding global piece slot ^ swz(token).
  auto issue_tile = [&](int tile, int buf) {
    const int t0 = tok0 + tile * kTok;
#pragma unroll
    for (int i = 0; i < LOADS_PER_WAVE; ++i) {
      const int P = (w * LOADS_PER_WAVE + i) * 64 + lane;
      const int tk = P / PK, slot = P % PK;
      const int tg = min(t0 + tk, tok1 - 1);
      const uint16_t* src = fbase + (size_t)tg * a.d + ((slot ^ swz(tk)) * 8);
      unsigned char* dst = &tile_buf[buf][(w * LOADS_PER_WAVE + i) * 64 * 16];
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)src, (lds_void*)dst, 16, 0, 0);
    }
  };

  const float sl2 = a.scale_log2;
  if (ntiles > 0) issue_tile(0, 0);
  for (int it = 0; it < ntiles; ++it) {
    const int cur = it & 1;
    if (it + 1 < ntiles) {
      issue_tile(it + 1, cur ^ 1);
      // wait for this wave's copies of tile `it`, leave the next tile in flight
      constexpr int N = LOADS_PER_WAVE;
      __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
    } else {
      __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0)
    }
    __syncthreads();
    const unsigned char* tb = tile_buf[cur];
    const int t0 = tok0 + it * kTok;

    // S^T = F_V Cq^T for the 4 16-token blocks of the tile
    floatx4 s[4][4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int tk = kb * 16 + c;
      bf16x8 xf[DC];
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = *reinterpret_cast<const u32x4*>(tb + tk * (DH * 2) + (((dc * 4 + G) ^ swz(tk)) * 16));
        xf[dc] = pk.b;
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dc = 0; dc < DC; ++dc) acc = mfma_bf16(xf[dc], qf[rb][dc], acc);
        s[kb][rb] = acc;
      }
    }

    // online softmax over the tile; P in fp16, ordered for the two 32-token halves
    f16x8 pf[2][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + kb * 16 + 4 * G + i;
          const float v = t < tok1 ? s[kb][rb][i] * sl2 : -INFINITY;
          s[kb][rb][i] = v;
          tmax = fmaxf(tmax, v);
        }
      tmax = wave_max_across_groups(tmax);
      const float mnew = fmaxf(m[rb], tmax);   // finite: every tile has a valid token
      const float alpha = exp2f(m[rb] - mnew);
      m[rb] = mnew;
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = exp2f(s[kb][rb][i] - mnew);
          psum += pv;
          pf[kb >> 1][rb][(kb & 1) * 4 + i] = (_Float16)pv;
        }
      l[rb] = l[rb] * alpha + psum;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
    }

    // O^T += F_V^T P^T with transposed fragments from LDS
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int tka = hf * 32 + 4 * G + (c >> 2);
      const int tkb = tka + 16;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int ch = db * 16 + 4 * (c & 3);       // channel of this lane's 8-byte read
        const int pc = ch >> 3, sub = (ch & 7) * 2;  // piece and byte offset inside it
        const unsigned char* pa = tb + tka * (DH * 2) + ((pc ^ swz(tka)) * 16) + sub;
        const unsigned char* pb = tb + tkb * (DH * 2) + ((pc ^ swz(tkb)) * 16) + sub;
        const shortx4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_shortx4*)((__attribute__((address_space(3))) unsigned char*)pa));
        const shortx4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_shortx4*)((__attribute__((address_space(3))) unsigned char*)pb));
        uint32_t w4[4];
        w4[0] = cvt_bf16x2_to_f16x2((uint32_t)(uint16_t)v0[0] | ((uint32_t)(uint16_t)v0[1] << 16));
        w4[1] = cvt_bf16x2_to_f16x2((uint32_t)(uint16_t)v0[2] | ((uint32_t)(uint16_t)v0[3] << 16));
        w4[2] = cvt_bf16x2_to_f16x2((uint32_t)(uint16_t)v1[0] | ((uint32_t)(uint16_t)v1[1] << 16));
        w4[3] = cvt_bf16x2_to_f16x2((uint32_t)(uint16_t)v1[2] | ((uint32_t)(uint16_t)v1[3] << 16));
        Pack8 vt;
        vt.u = u32x4{w4[0], w4[1], w4[2], w4[3]};
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) o[rb][db] = mfma_f16(vt.h, pf[hf][rb], o[rb][db]);
      }
    }
    __syncthreads();   // the buffer is refilled two tiles later
  }

  // normalise and write (directly, or as a partial for the merge)
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const float lt_ = wave_sum_across_groups(l[rb]);
    const int r = lat0 + rb * 16 + c;
    if (r >= a.C) continue;
    const float inv = lt_ > 0.f ? 1.f / lt_ : 0.f;
    if (nsplit == 1) {
      float* dst = a.out + ((size_t)b * a.C + r) * a.d + h * DH;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<floatx4*>(dst + db * 16 + 4 * G) = o[rb][db] * inv;
    } else {
      const size_t pr = ((size_t)bh * nsplit + split) * a.C + r;
      float* dst = a.part_o + pr * DH;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<floatx4*>(dst + db * 16 + 4 * G) = o[rb][db] * inv;
      if (G == 0) a.part_lse[pr] = lt_ > 0.f ? m[rb] + log2f(lt_) : -INFINITY;
    }
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
  switch (p.lat_tile / 64) {
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
    const int waves = std::min(4, (C + 63) / 64);
    p.lat_tile = waves * 64;
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
