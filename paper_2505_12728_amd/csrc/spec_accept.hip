// Speculative acceptance with residual resampling (SpecFLASH Sec. 3.1 and
// Sec. 3.3; greedy verification at temperature 0, Sec. 4.2).
//
// One 1024-thread work-group per sequence.  The vocabulary is cut into 16
// contiguous segments, one per wave; inside a segment the 64 lanes read
// consecutive entries, so every pass is a coalesced stream.
//
// Sampled mode
//   1. the k acceptance tests u_i q_i(x_i) < p_i(x_i) are exact float64
//      products of 24-bit significands; a ballot over the first k lanes and
//      a count of trailing ones give n;
//   2. fixed-point weights R_v = floor(r_v 2^40) of the residual
//      r = max(0, p_n - q_n) (one float32 subtraction) or of p_k;
//      per-wave uint64 sums, then the total S (exact: no rounding, so the
//      order of the additions does not matter);
//   3. T = floor(a S / 2^24) from the 24-bit uniform a = u_k 2^24, formed as
//      a (S >> 24) + ((a (S mod 2^24)) >> 24) without overflow;
//   4. the wave whose segment holds T rescans it with 64-wide inclusive
//      prefix sums and the first lane whose prefix exceeds T names the token.
// Greedy mode: a block-wide (value, lowest index) argmax per target row,
// row by row until the first draft that differs.
#include <math.h>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)v, m, 64);
  const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
  const uint32_t lo = __shfl_up((uint32_t)v, d, 64);
  const uint32_t hi = __shfl_up((uint32_t)(v >> 32), d, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v += shfl_xor_u64(v, m);
  return v;
}

// floor(r * 2^40) for r in [0, 1]: the scaling is exact in float32 and the
// conversion truncates.
__device__ __forceinline__ uint64_t fixed_weight(float r) {
  const float s = r * 1099511627776.0f;   // 2^40
  return s >= 1.0f ? (uint64_t)s : 0ull;
}

// Weight of entry v of the row being sampled.
// mode 0: max(0, p - q); mode 1: p alone.
__device__ __forceinline__ uint64_t weight_at(const float* prow, const float* qrow, int v,
                                              int use_q) {
  float r = prow[v];
  if (use_q) r = fmaxf(0.0f, r - qrow[v]);
  r = fmaxf(r, 0.0f);
  return fixed_weight(r);
}

struct Segment {
  int begin, end;
};

__device__ __forceinline__ Segment wave_segment(int w, int V) {
  const int per = ((V + kWaves - 1) / kWaves + 63) / 64 * 64;
  Segment s;
  s.begin = min(V, w * per);
  s.end = min(V, s.begin + per);
  return s;
}

// Exact total of the row's weights; per-wave totals land in wsum[].
__device__ uint64_t weight_total(const float* prow, const float* qrow, int use_q, int V,
                                 uint64_t* wsum) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const Segment sg = wave_segment(w, V);
  uint64_t acc = 0;
  int v = sg.begin + lane;
#pragma unroll 4
  for (; v < sg.end; v += 64) acc += weight_at(prow, qrow, v, use_q);
  acc = wave_sum_u64(acc);
  if (lane == 0) wsum[w] = acc;
  __syncthreads();
  uint64_t total = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) total += wsum[i];
  return total;
}

// Smallest j with sum_{v<=j} R_v > T (requires T < total).
__device__ int find_token(const float* prow, const float* qrow, int use_q, int V,
                          const uint64_t* wsum, uint64_t T, int* result) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint64_t before = 0;
  for (int i = 0; i < w; ++i) before += wsum[i];
  if (wsum[w] != 0 && before <= T && T < before + wsum[w]) {
    const Segment sg = wave_segment(w, V);
    uint64_t running = before;
    for (int v0 = sg.begin; v0 < sg.end; v0 += 64) {
      const int v = v0 + lane;
      uint64_t x = v < sg.end ? weight_at(prow, qrow, v, use_q) : 0ull;
      // inclusive 64-lane prefix sum
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint64_t y = shfl_up_u64(x, d);
        if (lane >= d) x += y;
      }
      const bool hit = running + x > T;
      const uint64_t mask = __ballot(hit);
      if (mask != 0ull) {
        if (lane == 0) *result = v0 + __builtin_ctzll(mask);
        break;
      }
      running += __shfl(x, 63, 64);
    }
  }
  __syncthreads();
  return *result;
}

// argmax over a row of float32 values, lowest index on ties.
__device__ int block_argmax(const float* row, int V, float* sval, int* sidx) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  for (int v = threadIdx.x; v < V; v += kThreads) {
    const float x = row[v];
    if (x > best || bi == 0x7fffffff) {   // indices increase, so ties keep the first
      best = x;
      bi = v;
    }
  }
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    const float ob = __shfl_xor(best, m, 64);
    const int oi = __shfl_xor(bi, m, 64);
    if (ob > best || (ob == best && oi < bi)) {
      best = ob;
      bi = oi;
    }
  }
  if (lane == 0) {
    sval[w] = best;
    sidx[w] = bi;
  }
  __syncthreads();
  float fb = sval[0];
  int fi = sidx[0];
  for (int i = 1; i < kWaves; ++i) {
    if (sval[i] > fb || (sval[i] == fb && sidx[i] < fi)) {
      fb = sval[i];
      fi = sidx[i];
    }
  }
  __syncthreads();   // sval / sidx are reused by the next call
  return fi;
}

__global__ __launch_bounds__(kThreads) void spec_accept_kernel(AcceptArgs a) {
  __shared__ uint64_t wsum[kWaves];
  __shared__ float sval[kWaves];
  __shared__ int sidx[kWaves];
  __shared__ int s_n;
  __shared__ int s_tok;
  const int b = blockIdx.x;
  const int k = a.k, V = a.V;
  const float* p = a.p + (size_t)b * (k + 1) * V;
  const int32_t* draft = a.draft + (size_t)b * k;
  int n = 0;
  int token = 0;

  if (a.mode == 0) {
    // greedy: longest prefix of drafts equal to the target argmax
    for (;;) {
      const int gi = block_argmax(p + (size_t)n * V, V, sval, sidx);
      if (n < k && draft[n] == gi) {
        ++n;
        continue;
      }
      token = gi;
      break;
    }
  } else {
    const float* q = a.q + (size_t)b * k * V;
    const float* u = a.u + (size_t)b * (k + 1);
    if (threadIdx.x < 64) {
      const int i = threadIdx.x;
      bool acc = false;
      if (i < k) {
        const int x = draft[i];
        if (x >= 0 && x < V) {
          const double pu = (double)u[i] * (double)q[(size_t)i * V + x];
          acc = pu < (double)p[(size_t)i * V + x];
        }
      }
      // bit i set where position i rejects; position k always "rejects"
      const uint64_t rej = __ballot(!acc) | (1ull << k);
      if (i == 0) s_n = __builtin_ctzll(rej);
    }
    __syncthreads();
    n = s_n;
    const float* prow = p + (size_t)n * V;
    const float* qrow = n < k ? q + (size_t)n * V : nullptr;
    int use_q = n < k ? 1 : 0;
    uint64_t S = weight_total(prow, qrow, use_q, V, wsum);
    if (S == 0 && use_q) {
      __syncthreads();
      use_q = 0;
      S = weight_total(prow, nullptr, 0, V, wsum);
    }
    if (S == 0) {
      token = block_argmax(prow, V, sval, sidx);
    } else {
      float uf = u[k] * 16777216.0f;   // exact: u is a float32
      uf = fminf(fmaxf(floorf(uf), 0.0f), 16777215.0f);
      const uint64_t av = (uint64_t)uf;
      const uint64_t T = av * (S >> 24) + ((av * (S & 0xffffffull)) >> 24);
      if (threadIdx.x == 0) s_tok = 0;
      __syncthreads();
      token = find_token(prow, qrow, use_q, V, wsum, T, &s_tok);
    }
  }

  int32_t* tok = a.tokens + (size_t)b * (k + 1);
  for (int i = threadIdx.x; i <= k; i += kThreads) {
    tok[i] = i < n ? draft[i] : (i == n ? token : -1);
  }
  if (threadIdx.x == 0) a.n_accepted[b] = n;
}

}  // namespace

hipError_t launch_accept(const AcceptArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(spec_accept_kernel, dim3(a.B), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace sd
