// One step of the draft's semi-autoregressive layer (SpecFLASH Sec. 3.1
// and Algorithm 1: the textual input FC(concat(F_T, E)); Sec. 3.3: one pass
// of one transformer layer gives the K placeholder states; Sec. 4.3: one
// layer of 32 heads):
//   x0 = [F_T, E] W_fc^T + b_fc
//   x1 = x0 + Attn(RoPE(RMSNorm(x0) Wqkv^T)) Wo^T      (cached context)
//   out = x1 + (silu(h Wg^T) * (h Wu^T)) Wdown^T,  h = RMSNorm(x1)
// for the r new rows of each sequence, over the draft's KV cache.
//
// A drafting step has few rows (R = B r <= 128 per pass), so every
// projection streams its weight once and is bound by HBM.  One kernel
// serves all five: work-groups of eight waves, 4..8 of which own 16 output
// columns each, and a range of 256-channel chunks of the reduction; lane
// (c, G) of a wave reads 128 contiguous bytes of weight row c per chunk
// (every row in 512-byte runs) straight into registers, the chunk of all
// input rows is copied into LDS by the global_load_lds DMA, and
// z^T = W x^T runs on bf16 matrix cores.  A compute unit streams weights at
// a bounded rate, so the planner sizes the column groups and reduction
// splits to give every unit the same load; each split writes fp32 partial
// sums, and one or two epilogue launches per projection add the splits
// and apply what follows it: bias + RMSNorm, RoPE + cache append, residual
// + RMSNorm, SwiGLU, or the final residual.  The attention is the
// verification kernel (its merge writing the bf16 input of Wo): the new
// rows are a block of r queries, causal inside the block, over the cache.
#include <math.h>

#include <algorithm>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;

constexpr int kChunkK = 256;    // reduction channels per step
constexpr int kEpiThreads = 256;

// part[ks][r][n] = sum over split ks's chunks of x[r][k] w[n][k], for the
// rows r0 .. r0 + 16 RB - 1 of this pass.  Matrix-core product i of a chunk
// takes the i-th 16-byte load of every lane (channels 64 G + 8 i .. +7 of
// the chunk), a fixed permutation of the chunk's channels that the input
// fragments follow; the input chunk's 16-byte pieces of row t sit at slot
// piece ^ (t & 15), so the fragment reads are free of bank conflicts.
// Two int8 values (bytes k, k + 1 of v) as two bf16 values, exactly (every
// int8 value has at most 8 significant bits): sign-extend, convert to
// float32, keep the upper halves.
__device__ __forceinline__ uint32_t i8x2_to_bf16x2(uint32_t v, int k) {
  const float f0 = (float)(int)(int8_t)(v >> (8 * k));
  const float f1 = (float)(int)(int8_t)(v >> (8 * k + 8));
  return __builtin_amdgcn_perm(__float_as_uint(f1), __float_as_uint(f0), 0x07060302u);
}

// Q8: the weight holds int8 rows with one fp32 scale per row (output
// column); each lane then loads 64 bytes of its row per chunk (4 loads),
// widens them to bf16 in registers and scales the accumulators once.
// A work-group owns a.cols = 16 x (active waves) output columns; waves past
// them only copy their share of the input chunks and meet the barriers, so
// the planner can size the groups to fill every compute unit evenly.
template <int RB, int NW, bool Q8>
__global__ __launch_bounds__(NW * 64) void linear_partial(LinearArgs a) {
  constexpr int HROWS = RB * 16;
  constexpr int HPIECES = HROWS * 32;          // 16-byte pieces of one input chunk
  constexpr int DMA = HPIECES / (NW * 64);     // copies per thread and chunk
  static_assert(HPIECES % (NW * 64) == 0, "whole copies per thread");
  __shared__ __align__(16) unsigned char hbuf[2][HPIECES * 16];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), G = lane >> 4, c = lane & 15;
  const int n0 = blockIdx.x * a.cols + w * 16;
  const bool active = w * 16 < a.cols;         // wave-uniform
  const int ks = blockIdx.y;
  const int r0 = blockIdx.z * HROWS;
  const int K = a.K, N = a.N, R = a.R;
  const int nch = K / kChunkK;
  const int ch0 = (int)((long long)nch * ks / a.ksplit);
  const int ch1 = (int)((long long)nch * (ks + 1) / a.ksplit);
  const uint16_t* W = static_cast<const uint16_t*>(a.w);
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  // weight row n0 + c (clamped; columns >= N are not written)
  const u32x4* wsrc = Q8 ? reinterpret_cast<const u32x4*>(static_cast<const int8_t*>(a.w) +
                                                          (size_t)min(n0 + c, N - 1) * K + 64 * G)
                         : reinterpret_cast<const u32x4*>(W + (size_t)min(n0 + c, N - 1) * K + 64 * G);
  constexpr int WL = Q8 ? 4 : 8;               // 16-byte weight loads per lane and chunk
  // copy j of this thread moves piece P = (w DMA + j) 64 + lane of a chunk:
  // input row P / 32 of the pass (clamped; padded rows are not written)
  const uint16_t* hsrc[DMA];
#pragma unroll
  for (int j = 0; j < DMA; ++j) {
    const int P = (w * DMA + j) * 64 + lane;
    const int row = P >> 5, slot = P & 31;
    hsrc[j] = X + (size_t)min(r0 + row, R - 1) * K + ((slot ^ (row & 15)) * 8);
  }
  auto issue = [&](int n, int buf) {
#pragma unroll
    for (int j = 0; j < DMA; ++j)
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)(hsrc[j] + (size_t)n * kChunkK),
                                       (lds_void*)(&hbuf[buf][(w * DMA + j) * 1024]), 16, 0, 0);
  };

  floatx4 acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = floatx4{0.f, 0.f, 0.f, 0.f};
  // the weights of chunk n + 1 are loaded before chunk n is multiplied, so
  // two chunks of every lane's row are in flight
  auto wload = [&](u32x4 (&wf)[WL], int n) {
#pragma unroll
    for (int i = 0; i < WL; ++i) wf[i] = wsrc[(size_t)n * (4 * WL) + i];
  };
  auto step = [&](const u32x4 (&wf)[WL], u32x4 (&wnext)[WL], int n) {
    const int buf = (n - ch0) & 1;
    if (n + 1 < ch1) {
      wload(wnext, n + 1);
      // the next weights are the WL newest loads: this thread's copies of
      // chunk n (and its weights) have landed; after the barrier every
      // wave's have, and every wave is done reading the other buffer
      wait_vm_then_barrier<WL>();
    } else {
      wait_vm_then_barrier<0>();
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      Pack8 x;
      if constexpr (Q8) {
        // product i takes bytes 8 (i & 1) .. + 7 of load i / 2: channels
        // 64 G + 8 i .. + 7 as in the bf16 layout
        const u32x4& v = wf[i >> 1];
        const uint32_t lo = v[(i & 1) * 2], hi = v[(i & 1) * 2 + 1];
        x.u = u32x4{i8x2_to_bf16x2(lo, 0), i8x2_to_bf16x2(lo, 2), i8x2_to_bf16x2(hi, 0), i8x2_to_bf16x2(hi, 2)};
      } else {
        x.u = wf[i];
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = rb * 16 + c;
        Pack8 y;
        y.u = *reinterpret_cast<const u32x4*>(&hbuf[buf][(row * 32 + ((8 * G + i) ^ c)) * 16]);
        acc[rb] = mfma_bf16(x.b, y.b, acc[rb]);
      }
    }
    if (n + 1 < ch1) issue(n + 1, buf ^ 1);
  };
  if (!active) {
    // input copies and barriers only, in the same order as the other waves
    if (ch0 < ch1) issue(ch0, 0);
#pragma unroll 1
    for (int n = ch0; n < ch1; ++n) {
      wait_vm_then_barrier<0>();
      if (n + 1 < ch1) issue(n + 1, ((n - ch0) & 1) ^ 1);
    }
    return;
  }
  u32x4 wa[WL], wb[WL];
  if (ch0 < ch1) {
    wload(wa, ch0);
    issue(ch0, 0);
  }
#pragma unroll 1
  for (int n = ch0; n < ch1; n += 2) {
    step(wa, wb, n);
    if (n + 1 < ch1) step(wb, wa, n + 1);
  }
  // accumulator element i of lane (c, G): input row rb*16 + c, column n0 + 4G + i
  if constexpr (Q8) {
    floatx4 sc;
#pragma unroll
    for (int i = 0; i < 4; ++i) sc[i] = a.wscale[min(n0 + 4 * G + i, N - 1)];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] *= sc;
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = r0 + rb * 16 + c;
    if (r >= R || n0 + 4 * G >= N) continue;
    float* dst = a.part + ((size_t)ks * R + r) * N + n0 + 4 * G;
    if (n0 + 4 * G + 3 < N && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      *reinterpret_cast<floatx4*>(dst) = acc[rb];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (n0 + 4 * G + i < N) dst[i] = acc[rb][i];
    }
  }
}

__device__ __forceinline__ float split_sum(const float* part, int ksplit, size_t stride, size_t idx) {
  float s = 0.f;
  for (int ks = 0; ks < ksplit; ++ks) s += part[(size_t)ks * stride + idx];
  return s;
}

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  return t;
}

// y = sum of splits (+ bias) (+ residual), written as fp32 `out` [R, N];
// grid (ceil(N / kEpiCols), R), kEpiThreads threads of four columns each.
// Every split of a thread's columns is loaded before any is added (the
// splits are added in split order), so a row's partials stream from many
// compute units at once.  With `ss`, block x of row r also writes the sum
// of squares of its columns to ss[r * gridDim.x + x] for epi_norm_cols.
constexpr int kEpiCols = 4 * kEpiThreads;
__global__ __launch_bounds__(kEpiThreads) void epi_add_cols(const float* part, int ksplit, int R, int N,
                                                            const float* bias, const float* residual,
                                                            float* out, float* ss) {
  __shared__ float red[kEpiThreads / 64];
  const int r = blockIdx.y;
  const size_t stride = (size_t)R * N;
  const size_t row = (size_t)r * N;
  const int n0 = blockIdx.x * kEpiCols + threadIdx.x * 4;
  auto a16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool vec = (N & 3) == 0 && a16(part) && a16(out) && (!bias || a16(bias)) && (!residual || a16(residual));
  float s2 = 0.f;
  if (vec) {
    if (n0 < N) {
      floatx4 v[kLinearMaxSplits];
#pragma unroll
      for (int ks = 0; ks < kLinearMaxSplits; ++ks)
        if (ks < ksplit) v[ks] = *reinterpret_cast<const floatx4*>(part + ks * stride + row + n0);
      floatx4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < kLinearMaxSplits; ++ks)
        if (ks < ksplit) y += v[ks];
      if (bias) y += *reinterpret_cast<const floatx4*>(bias + n0);
      if (residual) y += *reinterpret_cast<const floatx4*>(residual + row + n0);
      *reinterpret_cast<floatx4*>(out + row + n0) = y;
      s2 = y[0] * y[0] + y[1] * y[1] + y[2] * y[2] + y[3] * y[3];
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + j;
      if (n >= N) break;
      float y = split_sum(part, ksplit, stride, row + n);
      if (bias) y += bias[n];
      if (residual) y += residual[row + n];
      out[row + n] = y;
      s2 += y * y;
    }
  }
  if (ss == nullptr) return;
  const float t = block_sum(s2, red);
  if (threadIdx.x == 0) ss[(size_t)r * gridDim.x + blockIdx.x] = t;
}

// h = y / sqrt(mean(y^2) + eps) * norm_w in bf16, for the rows epi_add_cols
// wrote with their block sums of squares (nblk per row, added in block
// order); same grid as epi_add_cols.
__global__ __launch_bounds__(kEpiThreads) void epi_norm_cols(const float* y, int N, const float* ss, int nblk,
                                                             const float* norm_w, float eps, __bf16* h) {
  const int r = blockIdx.y;
  float t = 0.f;
  for (int i = 0; i < nblk; ++i) t += ss[(size_t)r * nblk + i];
  const float inv = 1.f / sqrtf(t / (float)N + eps);
  const int n0 = blockIdx.x * kEpiCols + threadIdx.x * 4;
  const size_t row = (size_t)r * N;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + j;
    if (n < N) h[row + n] = float_to_bf16(y[row + n] * inv * norm_w[n]);
  }
}

static int epi_blocks(int N) { return (N + kEpiCols - 1) / kEpiCols; }

// Fused projection output of row r (sequence b = r / rows, j = r % rows,
// position p = pos[b] + j): query heads rotated into q [R, Hq, D] (bf16),
// key heads rotated and value heads copied into the caches at position p
// (skipped when p is outside 0 .. Lmax - 1).  Half-split pairs (i, i + D/2)
// turn by p theta^(-2i/D): the frequencies are formed once per work-group
// in float64, the angle p f in float64 is reduced to [-pi, pi] in float64,
// and only the sine and cosine of the reduced angle are taken in float32
// (an error of a few float32 ulp at any position).  Row 0 of each sequence
// also writes kv_len[b] = pos[b] + rows for the attention.
__global__ __launch_bounds__(kEpiThreads) void epi_rope_qkv(const float* part, int ksplit, int R, int N,
                                                            const int32_t* pos, int rows, int Hq, int Hkv,
                                                            int D, double log_theta, int Lmax, __bf16* q,
                                                            __bf16* kc, __bf16* vc, int32_t* kv_len) {
  __shared__ float2 rot[64];                   // (cos, sin) of each pair's angle
  const int r = blockIdx.y;
  const int b = r / rows, j = r - b * rows;
  const int p = pos[b] + j;
  const bool store = p >= 0 && p < Lmax;
  if (j == 0 && blockIdx.x == 0 && threadIdx.x == 0) kv_len[b] = pos[b] + rows;
  const size_t stride = (size_t)R * N;
  const int half = D / 2;
  if (threadIdx.x < half) {
    const double f = exp(-2.0 * (double)threadIdx.x / (double)D * log_theta);
    const double ang = (double)p * f;
    const double twopi = 6.283185307179586476925286766559;
    const float red = (float)(ang - twopi * rint(ang / twopi));
    float sn, cs;
    sincosf(red, &sn, &cs);
    rot[threadIdx.x] = make_float2(cs, sn);
  }
  __syncthreads();
  // thread t of the row: pair t (query and key heads), then value element
  // t - pairs
  const int pairs = (Hq + Hkv) * half;
  const int t = blockIdx.x * kEpiThreads + threadIdx.x;
  if (t < pairs) {
    const int hh = t / half, i = t - hh * half;
    const size_t base = (size_t)r * N + (size_t)hh * D;
    const float x0 = split_sum(part, ksplit, stride, base + i);
    const float x1 = split_sum(part, ksplit, stride, base + i + half);
    const float cs = rot[i].x, sn = rot[i].y;
    const float y0 = x0 * cs - x1 * sn, y1 = x1 * cs + x0 * sn;
    if (hh < Hq) {
      __bf16* dst = q + ((size_t)r * Hq + hh) * D;
      dst[i] = float_to_bf16(y0);
      dst[i + half] = float_to_bf16(y1);
    } else if (store) {
      __bf16* dst = kc + (((size_t)b * Lmax + p) * Hkv + (hh - Hq)) * D;
      dst[i] = float_to_bf16(y0);
      dst[i + half] = float_to_bf16(y1);
    }
  } else if (store && t < pairs + Hkv * D) {
    const int hv = (t - pairs) / D, e = (t - pairs) - hv * D;
    const float v = split_sum(part, ksplit, stride, (size_t)r * N + (size_t)(Hq + Hkv + hv) * D + e);
    vc[(((size_t)b * Lmax + p) * Hkv + hv) * D + e] = float_to_bf16(v);
  }
}

// act[r][i] = silu(g) * u with g, u the split sums of columns i and I + i
__global__ __launch_bounds__(kEpiThreads) void epi_swiglu(const float* part, int ksplit, int R, int I,
                                                          __bf16* act) {
  const int r = blockIdx.y;
  const int i = blockIdx.x * kEpiThreads + threadIdx.x;
  if (i >= I) return;
  const size_t N = 2 * (size_t)I;
  const size_t stride = (size_t)R * N;
  const float g = split_sum(part, ksplit, stride, (size_t)r * N + i);
  const float u = split_sum(part, ksplit, stride, (size_t)r * N + I + i);
  act[(size_t)r * I + i] = float_to_bf16(g / (1.f + expf(-g)) * u);
}

// ------------------------------------------------- K drafts in K / k' passes
// Before the head: the k' placeholder rows of a pass's output (rows
// r - k' .. r - 1 of each sequence) rounded to bf16 as the LM head's input
// rows (b, j), and this pass's uniforms u[b][t k' + j] gathered.
__global__ __launch_bounds__(kEpiThreads) void kp_prep(const float* out, int r, int kp, int d, const float* u,
                                                       int K, int t, __bf16* hid, float* ut) {
  const int row = blockIdx.x;
  const int b = row / kp, j = row - b * kp;
  const float* src = out + ((size_t)b * r + (r - kp + j)) * d;
  for (int e = threadIdx.x; e < d; e += kEpiThreads) hid[(size_t)row * d + e] = float_to_bf16(src[e]);
  if (threadIdx.x == 0) ut[row] = u[(size_t)b * K + (size_t)t * kp + j];
}

// After the draw: row (b, j)'s token and distribution to the outputs at
// draft t k' + j; with another pass to come, the next pass's rows of
// sequence b (the drafted token, concat(bf16(F'), E[token]), then a
// placeholder row) and its positions pos_out[b] = pos_in[b] + advance.
// Token ids outside the vocabulary read the nearest embedding row.
__global__ __launch_bounds__(kEpiThreads) void kp_post(const float* probs, const int32_t* tok, int kp, int K,
                                                       int t, int V, int d, const __bf16* hid, const __bf16* emb,
                                                       const __bf16* ph, int32_t* tokens, float* q, __bf16* unext,
                                                       const int32_t* pos_in, int advance, int32_t* pos_out,
                                                       int more) {
  const int row = blockIdx.x;
  const int b = row / kp, j = row - b * kp;
  const int token = tok[row];
  const size_t dst = (size_t)b * K + (size_t)t * kp + j;
  if (threadIdx.x == 0) tokens[dst] = token;
  const float* src = probs + (size_t)row * V;
  float* qd = q + dst * V;
  for (int v = threadIdx.x; v < V; v += kEpiThreads) qd[v] = src[v];
  if (!more) return;
  const int tk = min(max(token, 0), V - 1);
  __bf16* text = unext + ((size_t)b * 2 * kp + j) * 2 * d;
  __bf16* place = unext + ((size_t)b * 2 * kp + kp + j) * 2 * d;
  for (int e = threadIdx.x; e < d; e += kEpiThreads) {
    text[e] = hid[(size_t)row * d + e];
    text[d + e] = emb[(size_t)tk * d + e];
  }
  for (int e = threadIdx.x; e < 2 * d; e += kEpiThreads) place[e] = ph[e];
  if (j == 0 && threadIdx.x == 0) pos_out[b] = pos_in[b] + advance;
}

template <int NW, bool Q8>
hipError_t launch_partial_nw(const LinearArgs& a, int rb, int passes, hipStream_t st) {
  const dim3 grid((a.N + a.cols - 1) / a.cols, a.ksplit, passes);
  const dim3 block(NW * 64);
  switch (rb) {
    case 1: hipLaunchKernelGGL((linear_partial<1, NW, Q8>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((linear_partial<2, NW, Q8>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((linear_partial<3, NW, Q8>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((linear_partial<4, NW, Q8>), grid, block, 0, st, a); break;
    case 5: hipLaunchKernelGGL((linear_partial<5, NW, Q8>), grid, block, 0, st, a); break;
    case 6: hipLaunchKernelGGL((linear_partial<6, NW, Q8>), grid, block, 0, st, a); break;
    case 7: hipLaunchKernelGGL((linear_partial<7, NW, Q8>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((linear_partial<8, NW, Q8>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

// Work-groups of the bf16 projection kernel resident per compute unit, as
// the runtime computes them from its registers, LDS and waves (for eight-
// wave groups the registers bind: two per unit, where the LDS of two input
// chunks would hold three); 0 when the runtime cannot tell.
template <int NW>
int resident_per_cu(int rb) {
  const void* f = nullptr;
  switch (rb) {
    case 1: f = reinterpret_cast<const void*>(&linear_partial<1, NW, false>); break;
    case 2: f = reinterpret_cast<const void*>(&linear_partial<2, NW, false>); break;
    case 3: f = reinterpret_cast<const void*>(&linear_partial<3, NW, false>); break;
    case 4: f = reinterpret_cast<const void*>(&linear_partial<4, NW, false>); break;
    case 5: f = reinterpret_cast<const void*>(&linear_partial<5, NW, false>); break;
    case 6: f = reinterpret_cast<const void*>(&linear_partial<6, NW, false>); break;
    case 7: f = reinterpret_cast<const void*>(&linear_partial<7, NW, false>); break;
    default: f = reinterpret_cast<const void*>(&linear_partial<8, NW, false>); break;
  }
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, NW * 64, 0) != hipSuccess) return 0;
  return n;
}

}  // namespace

LinearPlan plan_linear(int R, int K, int N, int cus) {
  LinearPlan p{};
  const int rows = std::min(R, kLinearRowsPerPass);
  p.row_blocks = (rows + 15) / 16;
  p.passes = (R + kLinearRowsPerPass - 1) / kLinearRowsPerPass;
  // work-groups resident per compute unit: the runtime's figure, else the
  // LDS bound (two input chunks of row_blocks * 8 KB) and 32 waves
  const int lds_fit = (160 * 1024) / (p.row_blocks * 16 * 1024);
  auto resident = [&](int waves) {
    int per_cu = resident_per_cu<8>(p.row_blocks);
    if (per_cu <= 0) per_cu = std::max(1, std::min(lds_fit, 32 / waves));
    return (long long)std::max(cus, 1) * per_cu;
  };
  // eight waves per work-group, each chunk of the inputs copied once for
  // all of them
  p.waves = 8;
  const long long cap = resident(p.waves);
  const int nch = K / kChunkK;
  const long long ncu = std::max(cus, 1);
  // A compute unit streams its weight rows at a bounded rate, so the time
  // follows the most loaded unit: (work-groups it runs) x (rows x chunks
  // per work-group).  For 4..8 column-owning waves, split the reduction to
  // fill the resident slots in one round (at least four chunks per split)
  // and keep the count with the least such load; ties go to more waves
  // (more weight loads in flight per unit).  One wave fewer than eight
  // fills every unit evenly where 128-column groups would leave units with
  // one group less than others (57344 columns: 512 groups of 112 instead
  // of 448 of 128).
  long long best = -1;
  for (int nwa = 8; nwa >= 4; --nwa) {
    const long long g = (long long)((N + nwa * 16 - 1) / (nwa * 16)) * p.passes;
    long long ks = std::max(1LL, cap / g);
    ks = std::min<long long>(ks, std::max(1, nch / 4));
    ks = std::max(1LL, std::min<long long>(ks, kLinearMaxSplits));
    const long long per_cu = (g * ks + ncu - 1) / ncu;
    const long long load = (long long)nwa * ((nch + ks - 1) / ks) * per_cu;
    if (best < 0 || load < best) {
      best = load;
      p.cols = nwa * 16;
      p.ksplit = (int)ks;
    }
  }
  p.part_bytes = (size_t)p.ksplit * R * N * sizeof(float);
  return p;
}

hipError_t launch_linear_partial(const LinearArgs& args, const LinearPlan& p, hipStream_t st) {
  LinearArgs a = args;
  a.cols = p.cols;
  if (a.wscale != nullptr) return launch_partial_nw<8, true>(a, p.row_blocks, p.passes, st);
  return launch_partial_nw<8, false>(a, p.row_blocks, p.passes, st);
}

hipError_t launch_epi_add(const float* part, int ksplit, int R, int N, const float* bias, const float* residual,
                          float* out, hipStream_t st) {
  hipLaunchKernelGGL(epi_add_cols, dim3(epi_blocks(N), R), dim3(kEpiThreads), 0, st, part, ksplit, R, N, bias,
                     residual, out, (float*)nullptr);
  return hipGetLastError();
}

// ------------------------------------------------------- the whole layer
static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

SemiArPlan plan_semi_ar(int B, int r, int d, int Hq, int Hkv, int I, int Lmax, int cus) {
  SemiArPlan p{};
  const int R = B * r, D = d / Hq;
  const int nqkv = (Hq + 2 * Hkv) * D;
  p.fc = plan_linear(R, 2 * d, d, cus);
  p.qkv = plan_linear(R, d, nqkv, cus);
  p.o = plan_linear(R, Hq * D, d, cus);
  p.gu = plan_linear(R, d, 2 * I, cus);
  p.down = plan_linear(R, I, d, cus);
  p.verify = plan_verify(B, r, Hq, Hkv, D, Lmax, 1, cus);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align256(bytes); return o; };
  const size_t part = std::max({p.fc.part_bytes, p.qkv.part_bytes, p.o.part_bytes, p.gu.part_bytes,
                                p.down.part_bytes});
  p.off_part = take(part);
  p.off_x0 = take((size_t)R * d * 4);
  p.off_h = take((size_t)R * d * 2);
  p.off_q = take((size_t)R * Hq * D * 2);
  p.off_attn16 = take((size_t)R * Hq * D * 2);
  p.off_x1 = take((size_t)R * d * 4);
  p.off_act = take((size_t)R * I * 2);
  p.off_kvlen = take((size_t)B * 4);
  p.off_ss = take((size_t)R * epi_blocks(d) * 4);
  p.off_verify = take(p.verify.workspace_bytes);
  p.workspace_bytes = off;
  p.ok = p.verify.ok;
  return p;
}

hipError_t launch_semi_ar(const SemiArArgs& a, const SemiArPlan& p, hipStream_t st) {
  unsigned char* ws = static_cast<unsigned char*>(a.workspace);
  float* part = reinterpret_cast<float*>(ws + p.off_part);
  float* x0 = reinterpret_cast<float*>(ws + p.off_x0);
  __bf16* h = reinterpret_cast<__bf16*>(ws + p.off_h);
  __bf16* q = reinterpret_cast<__bf16*>(ws + p.off_q);
  __bf16* attn16 = reinterpret_cast<__bf16*>(ws + p.off_attn16);
  float* x1 = reinterpret_cast<float*>(ws + p.off_x1);
  __bf16* act = reinterpret_cast<__bf16*>(ws + p.off_act);
  int32_t* kv_len = reinterpret_cast<int32_t*>(ws + p.off_kvlen);
  float* ss = reinterpret_cast<float*>(ws + p.off_ss);
  const int R = a.B * a.r, d = a.d, D = d / a.Hq;
  const dim3 eg(epi_blocks(d), R);
  const int nqkv = (a.Hq + 2 * a.Hkv) * D;
  hipError_t e;
  auto lin = [&](const void* x, const void* w, const float* scale, int K, int N, const LinearPlan& lp) {
    LinearArgs la{x, w, part, R, K, N, lp.ksplit, scale};
    return launch_linear_partial(la, lp, st);
  };
  // x0 = FC(u), h = RMSNorm(x0)
  if ((e = lin(a.u, a.fc_w, a.fc_s, 2 * d, d, p.fc)) != hipSuccess) return e;
  hipLaunchKernelGGL(epi_add_cols, eg, dim3(kEpiThreads), 0, st, part, p.fc.ksplit, R, d, a.fc_b,
                     (const float*)nullptr, x0, ss);
  hipLaunchKernelGGL(epi_norm_cols, eg, dim3(kEpiThreads), 0, st, x0, d, ss, (int)eg.x, a.ln1, a.eps, h);
  // q, k, v with RoPE; k, v appended to the cache
  if ((e = lin(h, a.wqkv, a.wqkv_s, d, nqkv, p.qkv)) != hipSuccess) return e;
  const int rope_threads = (a.Hq + a.Hkv) * (D / 2) + a.Hkv * D;
  hipLaunchKernelGGL(epi_rope_qkv, dim3((rope_threads + kEpiThreads - 1) / kEpiThreads, R), dim3(kEpiThreads), 0, st, part, p.qkv.ksplit, R, nqkv, a.pos, a.r,
                     a.Hq, a.Hkv, D, log((double)a.theta), a.Lmax, q,
                     static_cast<__bf16*>(a.k_cache), static_cast<__bf16*>(a.v_cache), kv_len);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // attention of the r new rows over the cache, causal inside them
  VerifyArgs va{};
  va.q = q;
  va.kc = a.k_cache;
  va.vc = a.v_cache;
  va.kv_len = kv_len;
  va.page_table = nullptr;
  va.Lmax = a.Lmax;
  va.out = nullptr;
  va.out_bf16 = attn16;                        // the merge writes the bf16 input of Wo
  va.lse = nullptr;
  va.B = a.B;
  va.k = a.r;
  va.Hq = a.Hq;
  va.Hkv = a.Hkv;
  va.D = D;
  va.scale = 1.f / sqrtf((float)D);
  va.scale_log2 = va.scale * kLog2e;
  va.part_o = reinterpret_cast<float*>(ws + p.off_verify);
  va.part_lse = va.part_o + p.verify.part_rows * D;
  if ((e = launch_verify(va, p.verify, 1, st)) != hipSuccess) return e;
  // x1 = x0 + attn Wo^T, h = RMSNorm(x1)
  if ((e = lin(attn16, a.wo, a.wo_s, a.Hq * D, d, p.o)) != hipSuccess) return e;
  hipLaunchKernelGGL(epi_add_cols, eg, dim3(kEpiThreads), 0, st, part, p.o.ksplit, R, d,
                     (const float*)nullptr, x0, x1, ss);
  hipLaunchKernelGGL(epi_norm_cols, eg, dim3(kEpiThreads), 0, st, x1, d, ss, (int)eg.x, a.ln2, a.eps, h);
  // act = SwiGLU(h), out = x1 + act Wdown^T
  if ((e = lin(h, a.wgu, a.wgu_s, d, 2 * a.I, p.gu)) != hipSuccess) return e;
  hipLaunchKernelGGL(epi_swiglu, dim3((a.I + kEpiThreads - 1) / kEpiThreads, R), dim3(kEpiThreads), 0, st, part,
                     p.gu.ksplit, R, a.I, act);
  if ((e = lin(act, a.wdown, a.wdown_s, a.I, d, p.down)) != hipSuccess) return e;
  return launch_epi_add(part, p.down.ksplit, R, d, nullptr, x1, a.out, st);
}

}  // namespace sd

namespace sd {

SemiArDraftPlan plan_semi_ar_draft(int B, int r0, int d, int Hq, int Hkv, int I, int Lmax, int V, int K, int kp,
                                   int cus) {
  SemiArDraftPlan p{};
  p.first = plan_semi_ar(B, r0, d, Hq, Hkv, I, Lmax, cus);
  p.later = K > kp ? plan_semi_ar(B, 2 * kp, d, Hq, Hkv, I, Lmax, cus) : p.first;
  const int rmax = std::max(r0, 2 * kp), R = B * kp;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align256(bytes); return o; };
  p.off_layer = take(std::max(p.first.workspace_bytes, p.later.workspace_bytes));
  p.off_out = take((size_t)B * rmax * d * 4);
  p.off_unext = take((size_t)B * 2 * kp * 2 * d * 2);
  p.off_hid = take((size_t)R * d * 2);
  p.off_probs = take((size_t)R * V * 4);
  p.off_lmstats = take(lm_head_workspace_bytes(R, V));
  p.off_sample = take(accept_workspace_bytes(R, 0, V, 1));
  p.off_nacc = take((size_t)R * 4);
  p.off_ut = take((size_t)R * 4);
  p.off_tok = take((size_t)R * 4);
  p.off_pos = take((size_t)2 * B * 4);
  p.workspace_bytes = off;
  p.cus = cus;
  p.ok = p.first.ok && p.later.ok;
  return p;
}

hipError_t launch_semi_ar_draft(const SemiArDraftArgs& a, const SemiArDraftPlan& p, hipStream_t st) {
  unsigned char* ws = static_cast<unsigned char*>(a.workspace);
  float* out = reinterpret_cast<float*>(ws + p.off_out);
  __bf16* unext = reinterpret_cast<__bf16*>(ws + p.off_unext);
  __bf16* hid = reinterpret_cast<__bf16*>(ws + p.off_hid);
  float* probs = reinterpret_cast<float*>(ws + p.off_probs);
  float* ut = reinterpret_cast<float*>(ws + p.off_ut);
  int32_t* tok = reinterpret_cast<int32_t*>(ws + p.off_tok);
  int32_t* posbuf = reinterpret_cast<int32_t*>(ws + p.off_pos);
  const int B = a.layer.B, d = a.layer.d, kp = a.kp, R = B * kp;
  const int passes = a.K / kp;
  hipError_t e;
  for (int t = 0; t < passes; ++t) {
    SemiArArgs la = a.layer;
    la.r = t == 0 ? a.layer.r : 2 * kp;
    la.u = t == 0 ? a.layer.u : unext;
    la.pos = t == 0 ? a.layer.pos : posbuf + (t & 1) * B;
    la.out = out;
    la.workspace = ws + p.off_layer;
    if ((e = launch_semi_ar(la, t == 0 ? p.first : p.later, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(kp_prep, dim3(R), dim3(kEpiThreads), 0, st, out, la.r, kp, d, a.u, a.K, t, hid, ut);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    LmHeadArgs lh{};
    lh.hidden = hid;
    lh.weight = a.lm_w;
    lh.probs = probs;
    lh.R = R;
    lh.d = d;
    lh.V = a.V;
    lh.scale_log2 = kLog2e / a.temperature;
    lh.stats = reinterpret_cast<float*>(ws + p.off_lmstats);
    lh.cus = p.cus;
    if ((e = launch_lm_head(lh, 1, st)) != hipSuccess) return e;
    AcceptArgs sa{};
    sa.p = probs;
    sa.u = ut;
    sa.n_accepted = reinterpret_cast<int32_t*>(ws + p.off_nacc);
    sa.tokens = tok;
    sa.B = R;
    sa.k = 0;
    sa.V = a.V;
    sa.mode = 1;
    if ((e = launch_accept(sa, ws + p.off_sample, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(kp_post, dim3(R), dim3(kEpiThreads), 0, st, probs, tok, kp, a.K, t, a.V, d, hid,
                       static_cast<const __bf16*>(a.emb), static_cast<const __bf16*>(a.ph), a.tokens, a.q, unext,
                       la.pos, la.r - kp, posbuf + ((t + 1) & 1) * B, (int)(t + 1 < passes));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sd
