// LM head with temperature softmax (SpecFLASH Sec. 3.1: the head maps a
// feature to a distribution over the vocabulary; Sec. 3.3 and Algorithm 1:
// the draft's hidden states go through the target's frozen head; Sec. 4.2:
// temperature):
//   probs[r, v] = softmax_v(hidden[r] . weight[v] / tau)
//
// The pass is bound by streaming the weight [V, d] once (R <= 256 rows share
// every weight byte), so the two kernels are shaped around that stream:
// 1. logits.  z^T = W H^T on bf16 matrix cores, the lane owning one hidden
//    row; every wave covers its own vocabulary rows for all R hidden rows,
//    so each weight byte is read once.  The scaled logits s = z log2(e) / tau
//    are written to `probs` as fp32, with (max, sum of 2^(s - max)) pairs
//    of every row: one per work-group (its waves' blocks merged in LDS) or
//    one per 16-entry vocabulary block.
//    - `lm_logits_burst` (R <= 64, d % 256 == 0): 16 vocabulary rows per
//      wave read in 512-byte runs per row, straight into registers; the
//      hidden chunk of 256 channels of all rows staged through LDS by DMA;
//      one pair per row and work-group.
//    - `lm_logits_bf16` (the other shapes): 16 or 32 vocabulary rows per
//      wave read 128 bytes per row at a time, the next 64 channels in
//      flight while the current ones are multiplied; the hidden chunk of 64
//      channels staged through double-buffered, swizzled LDS.
// 2. normalisation: every work-group merges its row's pairs into (M, L)
//    (a few kilobytes, read from L2), then rewrites probs = 2^(s - M) / L
//    in place.
// The fp32 path computes the logits as float64 dot products (one thread
// per row and entry) and shares kernel 2.
#include <math.h>

#include <algorithm>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

struct Stat {
  float m, l;
};

__device__ __forceinline__ Stat merge(Stat x, Stat y) {
  if (y.m == -INFINITY) return x;
  if (x.m == -INFINITY) return y;
  const float m = fmaxf(x.m, y.m);
  return Stat{m, x.l * fast_exp2(x.m - m) + y.l * fast_exp2(y.m - m)};
}

// statistics of 16 values spread as 4 per lane over the lanes c, c+16,
// c+32, c+48 (one accumulator column); invalid entries are -inf
__device__ __forceinline__ Stat column_stat(const floatx4& s) {
  float m = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
  m = wave_max_across_groups(m);
  float l = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int i = 0; i < 4; ++i) l += fast_exp2(s[i] - m);
  }
  l = wave_sum_across_groups(l);
  return Stat{m, l};
}

// KVB 16-entry vocabulary blocks per wave (2, or 1 when the vocabulary is
// too small to give about four work-groups per compute unit otherwise)
template <int RB, int KVB>
__global__ __launch_bounds__(256) void lm_logits_bf16(LmHeadArgs a) {
  constexpr int kVB = KVB;
  constexpr int kTileV = 4 * kVB * 16;             // vocabulary entries per work-group
  constexpr int HROWS = RB * 16;                   // hidden rows (padded)
  constexpr int HPIECES = HROWS * 8;               // 16-byte pieces of a 64-channel chunk
  constexpr int HPT = (HPIECES + 255) / 256;       // pieces staged per thread
  // hidden chunk (64 channels of every row), double-buffered; the 16-byte
  // pieces of row r sit at slot p ^ lds_swizzle<8>(r)
  __shared__ __align__(16) uint16_t hbuf[2][HROWS * 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, G = lane >> 4, c = lane & 15;
  const int v0 = blockIdx.x * kTileV + w * kVB * 16;   // this wave's first vocabulary row
  const int d = a.d, V = a.V, R = a.R;
  const uint16_t* W = static_cast<const uint16_t*>(a.weight);
  const uint16_t* H = static_cast<const uint16_t*>(a.hidden);
  // weight fragments: vocabulary row v0 + vb*16 + c (clamped; its results
  // are discarded), channels k + 8G .. k + 8G + 7 of each 32-channel step
  const u32x4* wsrc[kVB];
#pragma unroll
  for (int vb = 0; vb < kVB; ++vb)
    wsrc[vb] = reinterpret_cast<const u32x4*>(W + (size_t)min(v0 + vb * 16 + c, V - 1) * d + 8 * G);

  floatx4 acc[kVB][RB];
#pragma unroll
  for (int vb = 0; vb < kVB; ++vb)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = floatx4{0.f, 0.f, 0.f, 0.f};

  // the hidden chunk at channel k: this thread's pieces, global -> registers
  u32x4 hreg[HPT];
  auto h_load = [&](int k) {
#pragma unroll
    for (int i = 0; i < HPT; ++i) {
      const int P = i * 256 + tid;
      if (P < HPIECES) {
        const int row = min(P >> 3, R - 1);
        hreg[i] = *reinterpret_cast<const u32x4*>(H + (size_t)row * d + k + (P & 7) * 8);
      }
    }
  };
  auto h_store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < HPT; ++i) {
      const int P = i * 256 + tid;
      if (P < HPIECES) {
        const int row = P >> 3;
        *reinterpret_cast<u32x4*>(&hbuf[buf][(row * 8 + ((P & 7) ^ lds_swizzle<8>(row))) * 8]) = hreg[i];
      }
    }
  };
  // the weight chunk at channel k (two 32-channel steps)
  auto w_load = [&](u32x4 (&wf)[2][kVB], int k) {
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int vb = 0; vb < kVB; ++vb) wf[st][vb] = wsrc[vb][(k + 32 * st) / 8];
  };
  auto mma = [&](const u32x4 (&wf)[2][kVB], int buf) {
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = rb * 16 + c;
        Pack8 y;
        y.u = *reinterpret_cast<const u32x4*>(&hbuf[buf][(row * 8 + ((st * 4 + G) ^ lds_swizzle<8>(row))) * 8]);
#pragma unroll
        for (int vb = 0; vb < kVB; ++vb) {
          Pack8 x;
          x.u = wf[st][vb];
          acc[vb][rb] = mfma_bf16(x.b, y.b, acc[vb][rb]);
        }
      }
    }
  };

  // chunks of 64 channels: weight double-buffered in registers, hidden in LDS
  u32x4 wa[2][kVB], wb[2][kVB];
  w_load(wa, 0);
  h_load(0);
  h_store(0);
  __syncthreads();
  int k = 0;
#pragma unroll 1
  for (; k + 128 <= d; k += 128) {
    w_load(wb, k + 64);
    h_load(k + 64);
    mma(wa, 0);
    h_store(1);
    __syncthreads();   // chunk k+64 staged; every wave is done with buffer 0
    const bool more = k + 128 < d;
    if (more) {
      w_load(wa, k + 128);
      h_load(k + 128);
    }
    mma(wb, 1);
    if (more) h_store(0);
    __syncthreads();   // chunk k+128 staged; every wave is done with buffer 1
  }
  if (k < d) mma(wa, 0);   // d % 128 == 64: one chunk left

  // scaled logits, per-block statistics, fp32 logits to probs
  float2* stats = reinterpret_cast<float2*>(a.stats);
  const int nblk = (V + 15) / 16;
#pragma unroll
  for (int vb = 0; vb < kVB; ++vb) {
    const int vbase = v0 + vb * 16;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      floatx4 s;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = vbase + 4 * G + i;
        s[i] = v < V ? acc[vb][rb][i] * a.scale_log2 : -INFINITY;
      }
      const Stat st = column_stat(s);
      const int r = rb * 16 + c;
      if (r < R && vbase < V) {
        float* dst = a.probs + (size_t)r * V + vbase + 4 * G;
        if (vbase + 4 * G + 3 < V && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
          *reinterpret_cast<floatx4*>(dst) = s;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (vbase + 4 * G + i < V) dst[i] = s[i];
        }
        if (G == 0) stats[(size_t)r * nblk + vbase / 16] = make_float2(st.m, st.l);
      }
    }
  }
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_cvoid;

// Scaled logits of 16 vocabulary rows (accumulator rows) x 16 hidden rows
// (columns) to probs, with the (max, sum) of the 16-entry vocabulary block
// for every hidden row
template <bool STATS>
__device__ __forceinline__ Stat write_block(const LmHeadArgs& a, const floatx4& acc, int vbase, int r) {
  const int lane = threadIdx.x & 63, G = lane >> 4;
  const int V = a.V;
  floatx4 s;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = vbase + 4 * G + i;
    s[i] = v < V ? acc[i] * a.scale_log2 : -INFINITY;
  }
  const Stat st = column_stat(s);
  if (r < a.R && vbase < V) {
    float* dst = a.probs + (size_t)r * V + vbase + 4 * G;
    if (vbase + 4 * G + 3 < V && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      *reinterpret_cast<floatx4*>(dst) = s;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (vbase + 4 * G + i < V) dst[i] = s[i];
    }
    if (STATS && G == 0) reinterpret_cast<float2*>(a.stats)[(size_t)r * ((V + 15) / 16) + vbase / 16] = make_float2(st.m, st.l);
  }
  return st;
}

// Logits for R <= 64 hidden rows and widths d % 256 == 0, shaped for long
// contiguous weight reads.  Each wave owns VB blocks of 16 vocabulary rows;
// per chunk of 256 channels lane (c, G) loads 128 contiguous bytes of row c
// of each block (channels 64 G .. 64 G + 63) as eight back-to-back 16-byte
// loads, so every row is read in 512-byte runs (about 20% more HBM
// bandwidth than 128-byte runs on this weight layout).  Matrix-core product i takes the i-th load of every
// lane, i.e. channels {64 G + 8 i .. 64 G + 8 i + 7}: a fixed permutation of
// the chunk's channels, which the hidden fragments follow.  The hidden chunk
// of all rows (RB x 16 rows x 512 bytes) goes HBM/L2 -> LDS by the
// global_load_lds DMA into two buffers; pieces of row r sit at slot
// piece ^ (r & 15) so the 16 rows read at one piece hit 16 distinct bank
// groups.
//
// With a.nfull >= 0 the first a.nfull work-groups give every wave its VB
// blocks and the later ones leave their last wave without blocks (it only
// moves its share of the hidden chunks): the grid then holds a whole number
// of work-groups per compute unit with the larger ones dispatched first, so
// no unit streams more than one 16-row block above the mean.
template <int RB, int NW, int VB>
__global__ __launch_bounds__(NW * 64) void lm_logits_burst(LmHeadArgs a) {
  constexpr int HROWS = RB * 16;
  constexpr int HPIECES = HROWS * 32;          // 16-byte pieces of one hidden chunk
  constexpr int DMA = HPIECES / (NW * 64);     // copies per thread and chunk
  static_assert(HPIECES % (NW * 64) == 0, "whole copies per thread");
  __shared__ __align__(16) unsigned char hbuf[2][HPIECES * 16];
  __shared__ Stat wst[NW][HROWS];              // per wave: its blocks' statistics of every hidden row
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), G = lane >> 4, c = lane & 15;
  const int wg = blockIdx.x;
  const bool full = a.nfull < 0 || wg < a.nfull;
  const int unit0 = full ? wg * NW : a.nfull * NW + (wg - a.nfull) * (NW - 1);
  const int v0 = (unit0 + w) * (VB * 16);
  const int d = a.d, V = a.V, R = a.R;
  const uint16_t* W = static_cast<const uint16_t*>(a.weight);
  const uint16_t* H = static_cast<const uint16_t*>(a.hidden);
  // row c of each block of this wave (clamped; results of rows >= V are
  // discarded)
  const u32x4* wsrc[VB];
#pragma unroll
  for (int vb = 0; vb < VB; ++vb)
    wsrc[vb] = reinterpret_cast<const u32x4*>(W + (size_t)min(v0 + vb * 16 + c, V - 1) * d + 64 * G);
  // copy j of this thread moves piece P = (w * DMA + j) * 64 + lane of the
  // chunk: hidden row P / 32 (clamped; padded rows are discarded), LDS slot
  // P % 32 holding global piece slot ^ (row & 15)
  const uint16_t* hsrc[DMA];
#pragma unroll
  for (int j = 0; j < DMA; ++j) {
    const int P = (w * DMA + j) * 64 + lane;
    const int row = P >> 5, slot = P & 31;
    hsrc[j] = H + (size_t)min(row, R - 1) * d + ((slot ^ (row & 15)) * 8);
  }
  auto issue_hidden = [&](int n, int buf) {
#pragma unroll
    for (int j = 0; j < DMA; ++j)
      __builtin_amdgcn_global_load_lds((gbl_cvoid*)(hsrc[j] + n * 256),
                                       (lds_void*)(&hbuf[buf][(w * DMA + j) * 1024]), 16, 0, 0);
  };

  floatx4 acc[VB][RB];
#pragma unroll
  for (int vb = 0; vb < VB; ++vb)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nch = d / 256;
  issue_hidden(0, 0);
  const bool idle = !full && w == NW - 1;
  if (idle) {
    // same copies, waits and barriers as the other waves, no weight rows
#pragma unroll 1
    for (int n = 0; n < nch; ++n) {
      wait_vm_then_barrier<0>();
      if (n + 1 < nch) issue_hidden(n + 1, (n & 1) ^ 1);
    }
  } else {
#pragma unroll 1
  for (int n = 0; n < nch; ++n) {
    const int buf = n & 1;
    u32x4 wf[VB][8];
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int i = 0; i < 8; ++i) wf[vb][i] = wsrc[vb][n * 32 + i];
    // the weight loads are the newest: everything older (this thread's
    // copies of chunk n) has landed; after the barrier every wave's copies
    // have, and every wave is done reading the other buffer
    wait_vm_then_barrier<8 * VB>();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = rb * 16 + c;
        Pack8 y;
        y.u = *reinterpret_cast<const u32x4*>(&hbuf[buf][(row * 32 + ((8 * G + i) ^ c)) * 16]);
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) {
          Pack8 x;
          x.u = wf[vb][i];
          acc[vb][rb] = mfma_bf16(x.b, y.b, acc[vb][rb]);
        }
      }
    }
    if (n + 1 < nch) issue_hidden(n + 1, buf ^ 1);
  }
  }
  // scaled logits to probs; the statistics of this work-group's blocks,
  // merged over its waves, as one (max, sum) pair per hidden row at
  // stats[r * gridDim.x + blockIdx.x]
  Stat st[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) st[rb] = Stat{-INFINITY, 0.f};
  if (!idle) {
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) st[rb] = merge(st[rb], write_block<false>(a, acc[vb][rb], v0 + vb * 16, rb * 16 + c));
  }
  if (G == 0) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) wst[w][rb * 16 + c] = st[rb];
  }
  __syncthreads();
  if (tid < HROWS && tid < R) {
    Stat t = wst[0][tid];
#pragma unroll
    for (int i = 1; i < NW; ++i) t = merge(t, wst[i][tid]);
    reinterpret_cast<float2*>(a.stats)[(size_t)tid * gridDim.x + blockIdx.x] = make_float2(t.m, t.l);
  }
}

// fp32 inputs: one thread per (row, vocabulary entry), float64 dot product;
// 16 consecutive lanes form one 16-entry block for the statistics
__global__ __launch_bounds__(256) void lm_logits_f32(LmHeadArgs a) {
  const int r = blockIdx.y;
  const int v = blockIdx.x * 256 + threadIdx.x;
  const int d = a.d, V = a.V;
  const float* h = static_cast<const float*>(a.hidden) + (size_t)r * d;
  float s = -INFINITY;
  if (v < V) {
    const float* wr = static_cast<const float*>(a.weight) + (size_t)v * d;
    double z = 0.0;
    for (int j = 0; j < d; ++j) z += (double)h[j] * (double)wr[j];
    s = (float)(z * (double)a.scale_log2);
    a.probs[(size_t)r * V + v] = s;
  }
  float m = s;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  float l = m == -INFINITY ? 0.f : fast_exp2(s - m);
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) l += __shfl_xor(l, o, 64);
  const int nblk = (V + 15) / 16;
  if ((threadIdx.x & 15) == 0 && v < V)
    reinterpret_cast<float2*>(a.stats)[(size_t)r * nblk + v / 16] = make_float2(m, l);
}

// probs = 2^(s - M) / L, in place, 16-byte accesses when the row allows.
// Each work-group first merges the row's npairs (max, sum) pairs into
// (M, L), every thread taking its pairs eight at a time (eight loads in
// flight, then one rescale), so the merge costs a few memory latencies.
__global__ __launch_bounds__(256) void lm_normalize(LmHeadArgs a, int npairs) {
  __shared__ Stat part[4];
  const int r = blockIdx.y;
  const int V = a.V;
  const float2* st = reinterpret_cast<const float2*>(a.stats) + (size_t)r * npairs;
  Stat acc{-INFINITY, 0.f};
  for (int base = threadIdx.x; base < npairs; base += 256 * 8) {
    float2 x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = base + j * 256;
      x[j] = i < npairs ? st[i] : make_float2(-INFINITY, 0.f);
    }
    float m = acc.m;
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, x[j].x);
    if (m != -INFINITY) {
      float l = acc.l * fast_exp2(acc.m - m);
#pragma unroll
      for (int j = 0; j < 8; ++j) l += x[j].y * fast_exp2(x[j].x - m);
      acc = Stat{m, l};
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc = merge(acc, Stat{__shfl_xor(acc.m, o, 64), __shfl_xor(acc.l, o, 64)});
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  Stat ML = part[0];
#pragma unroll
  for (int i = 1; i < 4; ++i) ML = merge(ML, part[i]);
  const float inv = 1.f / ML.l;
  float* row = a.probs + (size_t)r * V;
  const int stride = gridDim.x * 256;
  if ((V & 3) == 0 && (reinterpret_cast<uintptr_t>(row) & 15) == 0) {
    // a contiguous range of 16-byte pieces per work-group, eight loads in
    // flight per thread before any store
    floatx4* row4 = reinterpret_cast<floatx4*>(row);
    const int n4 = V / 4, per = (n4 + gridDim.x - 1) / gridDim.x;
    const int c0 = blockIdx.x * per, c1 = min(n4, c0 + per);
    for (int base = c0 + threadIdx.x; base < c1; base += 256 * 8) {
      floatx4 x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (base + j * 256 < c1) x[j] = row4[base + j * 256];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (base + j * 256 < c1) {
#pragma unroll
          for (int i = 0; i < 4; ++i) x[j][i] = fast_exp2(x[j][i] - ML.m) * inv;
          row4[base + j * 256] = x[j];
        }
    }
  } else {
    for (int v = blockIdx.x * 256 + threadIdx.x; v < V; v += stride) row[v] = fast_exp2(row[v] - ML.m) * inv;
  }
}

// Launches the logits kernel; *npairs receives the statistics pairs it
// writes per row (one per work-group for the long-row kernel, one per
// 16-entry block otherwise).
template <int RB>
hipError_t launch_rb(const LmHeadArgs& a, hipStream_t st, int* npairs) {
  *npairs = (a.V + 15) / 16;
  if constexpr (RB <= 4) {
    if (a.d % 256 == 0) {
      LmHeadArgs b = a;
      b.nfull = -1;
      if (a.V >= 65536) {
        // G work-groups, a multiple of the unit count, of 8 or 7 blocks
        // (nfull = nb - 7 G of 8) when such a G covers the nb blocks
        const int nb = (a.V + 15) / 16, g8 = (nb + 7) / 8;
        int grid = g8;
        if (a.cus > 0) {
          const int G = (g8 + a.cus - 1) / a.cus * a.cus;
          if (G > g8 && 7LL * G <= nb) {
            grid = G;
            b.nfull = nb - 7 * G;
          }
        }
        hipLaunchKernelGGL((lm_logits_burst<RB, 8, 1>), dim3(grid), dim3(512), 0, st, b);
        *npairs = grid;
      } else {
        hipLaunchKernelGGL((lm_logits_burst<RB, 4, 1>), dim3((a.V + 63) / 64), dim3(256), 0, st, b);
        *npairs = (a.V + 63) / 64;
      }
      return hipGetLastError();
    }
  }
  if ((a.V + 127) / 128 >= 1024) {
    hipLaunchKernelGGL((lm_logits_bf16<RB, 2>), dim3((a.V + 127) / 128), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((lm_logits_bf16<RB, 1>), dim3((a.V + 63) / 64), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace

size_t lm_head_workspace_bytes(int R, int V) {
  const size_t nblk = ((size_t)V + 15) / 16;
  return ((size_t)R * nblk + (size_t)R) * sizeof(float2);
}

hipError_t launch_lm_head(const LmHeadArgs& a, int dtype, hipStream_t st) {
  hipError_t e = hipSuccess;
  int npairs = (a.V + 15) / 16;
  if (dtype == 0) {
    hipLaunchKernelGGL(lm_logits_f32, dim3((a.V + 255) / 256, a.R), dim3(256), 0, st, a);
    e = hipGetLastError();
  } else {
    switch ((a.R + 15) / 16) {
      case 1: e = launch_rb<1>(a, st, &npairs); break;
      case 2: e = launch_rb<2>(a, st, &npairs); break;
      case 3: e = launch_rb<3>(a, st, &npairs); break;
      case 4: e = launch_rb<4>(a, st, &npairs); break;
      case 5: e = launch_rb<5>(a, st, &npairs); break;
      case 6: e = launch_rb<6>(a, st, &npairs); break;
      case 7: e = launch_rb<7>(a, st, &npairs); break;
      case 8: e = launch_rb<8>(a, st, &npairs); break;
      case 9: e = launch_rb<9>(a, st, &npairs); break;
      case 10: e = launch_rb<10>(a, st, &npairs); break;
      case 11: e = launch_rb<11>(a, st, &npairs); break;
      case 12: e = launch_rb<12>(a, st, &npairs); break;
      case 13: e = launch_rb<13>(a, st, &npairs); break;
      case 14: e = launch_rb<14>(a, st, &npairs); break;
      case 15: e = launch_rb<15>(a, st, &npairs); break;
      case 16: e = launch_rb<16>(a, st, &npairs); break;
      default: return hipErrorInvalidValue;   // R <= 256 is checked by the caller
    }
  }
  if (e != hipSuccess) return e;
  // up to eight 16-byte pieces per thread: each work-group also reads the
  // row's pairs, so fewer, fuller work-groups read them fewer times; but
  // at least two work-groups per compute unit over all rows while that
  // leaves each thread two pieces or more
  const int cus = a.cus > 0 ? a.cus : 256;
  const int per_row = std::max((a.V + 8191) / 8192, std::min((a.V + 2047) / 2048, (2 * cus + a.R - 1) / a.R));
  hipLaunchKernelGGL(lm_normalize, dim3(std::min(per_row, 64), a.R), dim3(256), 0, st, a, npairs);
  return hipGetLastError();
}

}  // namespace sd
