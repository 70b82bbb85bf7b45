// Speculative acceptance with residual resampling (SpecFLASH Sec. 3.1 and
// Sec. 3.3; greedy verification at temperature 0, Sec. 4.2).
//
// One kernel, one work-group per (vocabulary chunk, sequence) on a 1-D grid
// (chunks fastest), 256 threads, in two phases:
//
// 1. chunk phase, every work-group.
//    Sampled mode: every work-group of a sequence repeats the k acceptance
//    tests u_i q_i(x_i) < p_i(x_i) (exact float64 products of 24-bit
//    significands; a ballot and a count of trailing ones give n), then sums
//    over its chunk the fixed-point weights of the row that will be sampled,
//    R_v = floor(r_v 2^40) with r = max(0, p_n - q_n) (one float32
//    subtraction) or r = p_k, and the fallback weights floor(p_n 2^40).
//    Integer sums are exact, so the order of additions does not matter.
//    Greedy mode: the (value, lowest index) maximum of every target row
//    over the chunk.
// 2. finish phase, in the last work-group of each sequence to complete its
//    chunk (an arrival counter per sequence in the workspace, counted with
//    a device-scope atomic once the work-group's partials are written with
//    device-scope stores; the last arrival resets it to zero, so a
//    workspace that starts zeroed stays valid for the next call), one
//    thread per chunk.
//    Sampled: a block prefix sum of the chunk sums gives S and each chunk's
//    starting offset; T = floor(a S / 2^24) from a = u_k 2^24 (formed as
//    a (S >> 24) + ((a (S mod 2^24)) >> 24) without overflow) picks the
//    chunk, and inside it the first entry whose inclusive prefix sum
//    exceeds T (the chunk's entries loaded in one round, four consecutive
//    ones per thread, and a block prefix sum of the threads' totals).
//    Greedy: argmax per row from the chunk maxima, then the longest
//    matching prefix.
// Every vocabulary access is a coalesced stream.
//
// From logits (the target's k + 1 and the draft's k rows per sequence), the
// same kernel reads p and q on demand as a temperature softmax of the
// logits, after a statistics pass, one work-group per (4096-entry chunk, row), that writes
// each chunk's (max, sum of 2^(z s - max)) with s = log2(e) / tau.  Each
// work-group of the rule first merges its sequence's 2k + 1 rows of chunk
// statistics into (M, 1 / L) in LDS.  The uniforms come from Philox-4x64-10
// on the device.  Greedy mode skips the statistics and compares the target
// logits directly.
#include <math.h>

#include "device_common.hpp"
#include "launch.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 1024;     // vocabulary entries per chunk (<= 256 chunks for V <= 2^18)
static_assert(kChunk % kThreads == 0, "whole entries per thread in a chunk");
constexpr int kStatChunk = 4096;
constexpr int kMaxStatParts = (1 << 18) / kStatChunk;   // statistics chunks of a row at most

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

// floor(r * 2^40) for r in [0, 1] (clamped there): the scaling is exact in
// float32 and the conversion truncates.
__device__ __forceinline__ uint64_t fixed_weight(float r) {
  r = fminf(fmaxf(r, 0.0f), 1.0f);
  const float s = r * 1099511627776.0f;   // 2^40
  return s >= 1.0f ? (uint64_t)s : 0ull;
}

// Where the rule's inputs come from.  A source gives, for sequence b,
// position i and token v: target(b, i, v) = p_i(v), drafted(b, i, v) =
// q_i(v), greedy(b, i, v) = the value whose row maximum is the greedy token,
// and uniform(b, i) = u_i.

// p, q and u handed over as float32 arrays
struct ProbSrc {
  const float* p;
  const float* q;
  const float* u;
  int k, V;
  __device__ __forceinline__ float target(int b, int i, int v) const {
    return p[((size_t)b * (k + 1) + i) * V + v];
  }
  __device__ __forceinline__ float drafted(int b, int i, int v) const {
    return q[((size_t)b * k + i) * V + v];
  }
  __device__ __forceinline__ float greedy(int b, int i, int v) const { return target(b, i, v); }
  __device__ __forceinline__ float uniform(int b, int i) const { return u[(size_t)b * (k + 1) + i]; }
  __device__ __forceinline__ void prepare(int, float2*) {}
};

// Philox-4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 64 x 64 -> 128-bit products, the high halves mixed with the other words
// and the key, the key bumped by the Weyl increments.  Uniform i of sequence
// b is word i % 4 of the block at counter (i / 4, b, offset, 0) under key
// (seed, 0), as a multiple of 2^-24: (word >> 40) * 2^-24.
__device__ __forceinline__ float philox_uniform(uint64_t seed, uint64_t offset, int b, int i) {
  uint64_t c0 = (uint64_t)(i >> 2), c1 = (uint64_t)b, c2 = offset, c3 = 0;
  uint64_t k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t lo0 = 0xD2E7470EE14C6C93ull * c0, hi0 = __umul64hi(0xD2E7470EE14C6C93ull, c0);
    const uint64_t lo1 = 0xCA5A826395121157ull * c2, hi1 = __umul64hi(0xCA5A826395121157ull, c2);
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  const int wsel = i & 3;
  const uint64_t word = wsel == 0 ? c0 : (wsel == 1 ? c1 : (wsel == 2 ? c2 : c3));
  return (float)(word >> 40) * 5.9604644775390625e-08f;   // 2^-24
}

__device__ __forceinline__ float load_logit(const float* z, size_t i) { return z[i]; }
__device__ __forceinline__ float load_logit(const uint16_t* z, size_t i) { return bf16_bits_to_float(z[i]); }

// p and q from logits at temperature tau: p_i(v) = 2^(z_i(v) s - M_i) / L_i
// with s = log2(e) / tau; u from Philox.  Greedy compares the target logits
// themselves.  `part` holds the chunk statistics (max, sum) of every row
// (target rows b (k+1) + i, then draft rows B (k+1) + b k + i);
// prepare(b) merges the 2k + 1 rows of sequence b into (M, 1 / L) in the
// work-group's LDS array `rows` (target rows 0..k, then draft rows), which
// target() and drafted() read.
template <typename T>
struct LogitSrc {
  const T* zt;
  const T* zd;
  const float2* part;
  int nparts;
  float2* rows;
  float s;
  uint64_t seed, offset;
  int B, k, V;
  __device__ __forceinline__ float target(int b, int i, int v) const {
    const float2 st = rows[i];
    return fast_exp2(load_logit(zt, ((size_t)b * (k + 1) + i) * V + v) * s - st.x) * st.y;
  }
  __device__ __forceinline__ float drafted(int b, int i, int v) const {
    const float2 st = rows[k + 1 + i];
    return fast_exp2(load_logit(zd, ((size_t)b * k + i) * V + v) * s - st.x) * st.y;
  }
  // Eight lanes per row, up to eight chunk partials each (nparts <= 64):
  // all loads issue at once, then a max and a rescaled sum over the eight
  // lanes.  The caller synchronises before reading `rows`.
  __device__ void prepare(int b, float2* lds) {
    rows = lds;
    if (part == nullptr) return;               // greedy: no statistics
    const int sub = threadIdx.x & 7;
    for (int j0 = 0; j0 <= 2 * k; j0 += kThreads / 8) {
      const int j = j0 + (int)(threadIdx.x >> 3);
      const bool live = j <= 2 * k;
      const size_t r = j <= k ? (size_t)b * (k + 1) + j : (size_t)B * (k + 1) + (size_t)b * k + (j - k - 1);
      const float2* pr = part + r * nparts;
      float2 v[kMaxStatParts / 8];
#pragma unroll
      for (int i = 0; i < kMaxStatParts / 8; ++i) {
        const int c = sub + 8 * i;
        v[i] = live && c < nparts ? pr[c] : make_float2(-INFINITY, 0.f);
      }
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < kMaxStatParts / 8; ++i) m = fmaxf(m, v[i].x);
#pragma unroll
      for (int o = 4; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      float l = 0.f;
#pragma unroll
      for (int i = 0; i < kMaxStatParts / 8; ++i)
        if (v[i].x != -INFINITY) l += v[i].y * fast_exp2(v[i].x - m);
#pragma unroll
      for (int o = 4; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
      if (live && sub == 0) lds[j] = make_float2(m, 1.f / l);
    }
  }
  __device__ __forceinline__ float greedy(int b, int i, int v) const {
    return load_logit(zt, ((size_t)b * (k + 1) + i) * V + v);
  }
  __device__ __forceinline__ float uniform(int b, int i) const { return philox_uniform(seed, offset, b, i); }
};

// Sampled weight of entry v of row n: residual (use_q) or p alone.
template <typename Src>
__device__ __forceinline__ uint64_t weight_at(const Src& src, int b, int n, int v, int use_q) {
  float r = src.target(b, n, v);
  if (use_q) r = fmaxf(0.0f, r - src.drafted(b, n, v));
  return fixed_weight(r);
}

// n for one sequence: leading accepted drafts.  Uses lanes 0..63 of wave 0;
// the result is returned to every thread through `slot`.
template <typename Src>
__device__ int accepted_prefix(const AcceptArgs& a, const Src& src, int b, int* slot, int* drafts) {
  const int k = a.k, V = a.V;
  if (threadIdx.x < 64) {
    const int i = threadIdx.x;
    bool acc = false;
    if (i < k) {
      const float ui = src.uniform(b, i);      // independent of the draft id: issued with it
      const int x = a.draft[(size_t)b * k + i];
      drafts[i] = x;
      if (x >= 0 && x < V) {
        const double pu = (double)ui * (double)src.drafted(b, i, x);
        acc = pu < (double)src.target(b, i, x);
      }
    }
    // bit i set where position i rejects; position k always "rejects"
    const uint64_t rej = __ballot(!acc) | (1ull << k);
    if (i == 0) *slot = __builtin_ctzll(rej);
  }
  __syncthreads();
  return *slot;
}

struct ArgMax {
  float v;
  int i;
};

__device__ __forceinline__ ArgMax better(ArgMax x, ArgMax y) {
  // larger value wins; equal values: lower index wins; i < 0 means empty
  if (y.i < 0) return x;
  if (x.i < 0) return y;
  if (y.v > x.v || (y.v == x.v && y.i < x.i)) return y;
  return x;
}

// (value, lowest index) maximum of value(v) over [v0, v1)
template <typename F>
__device__ ArgMax block_argmax_range(F&& value, int v0, int v1, ArgMax* sm) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  ArgMax best{-INFINITY, -1};
  for (int v = v0 + threadIdx.x; v < v1; v += kThreads) {
    const float x = value(v);
    if (best.i < 0 || x > best.v) best = ArgMax{x, v};   // indices increase: ties keep the first
  }
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    ArgMax o{__shfl_xor(best.v, m, 64), __shfl_xor(best.i, m, 64)};
    best = better(best, o);
  }
  if (lane == 0) sm[w] = best;
  __syncthreads();
  ArgMax r = sm[0];
  for (int i = 1; i < kWaves; ++i) r = better(r, sm[i]);
  __syncthreads();
  return r;
}

// workspace layout: arrival counters first, then the chunk partials
//   uint32 count[B][kCounterStride] (one counter per 128-byte line)
//   sampled: uint64 sums[B][C][2]  (residual / p-only)
//   greedy:  ArgMax best[B][k+1][C]
__host__ __device__ __forceinline__ size_t counter_bytes(int B) {
  return ((size_t)B * kCounterStride * sizeof(unsigned) + 255) / 256 * 256;
}

// Partials cross work-groups (possibly on other XCDs, behind other L2
// caches) as device-scope stores and loads of 64-bit words (publish /
// fetch_published).
__device__ __forceinline__ uint64_t load_partial(const uint64_t* p) { return fetch_published(p); }
__device__ __forceinline__ ArgMax load_partial(const ArgMax* p) {
  const uint64_t x = fetch_published(reinterpret_cast<const uint64_t*>(p));
  return ArgMax{__uint_as_float((uint32_t)x), (int)(uint32_t)(x >> 32)};
}
__device__ __forceinline__ void store_partial(ArgMax* p, ArgMax r) {
  publish(reinterpret_cast<uint64_t*>(p), ((uint64_t)(uint32_t)r.i << 32) | __float_as_uint(r.v));
}

constexpr int kMaxRows = 17;   // k + 1 rows at most (k <= 16)
constexpr int kPer = kChunk / kThreads;
constexpr int kRowGroup = 4;   // greedy rows reduced per barrier

struct RuleShared {
  uint64_t wsum[kWaves][2];
  uint64_t tot[kWaves];
  ArgMax sm[kWaves];
  ArgMax gsm[kRowGroup][kWaves];
  ArgMax gmax[kMaxRows];
  int drafts[kMaxRows];
  uint64_t before;
  int n, tok, chunk, last;
  float2 rows[33];
};

// Phase 1: this work-group's chunk partials of sequence b.  Thread t takes
// entries v0 + j kThreads + t (j < kPer); every load of a row is issued
// before any is used.
template <typename Src>
__device__ void chunk_phase(const AcceptArgs& a, const Src& src, unsigned char* parts, int nchunks, int chunk,
                            int b, RuleShared& sh) {
  const int k = a.k, V = a.V;
  const int v0 = chunk * kChunk, v1 = min(V, v0 + kChunk);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (a.mode == 0) {
    // (value, lowest index) maximum of every target row over the chunk,
    // kRowGroup rows at a time: all their loads in flight, wave maxima by
    // shuffles, one barrier, then one thread per row merges the waves
    ArgMax* out = reinterpret_cast<ArgMax*>(parts) + (size_t)b * (k + 1) * nchunks;
    float x[kMaxRows][kPer];                   // every row's loads in flight at once
#pragma unroll
    for (int r = 0; r < kMaxRows; ++r)
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const int v = v0 + j * kThreads + threadIdx.x;
        x[r][j] = (r <= k && v < v1) ? src.greedy(b, r, v) : 0.f;
      }
#pragma unroll
    for (int i0 = 0; i0 < kMaxRows; i0 += kRowGroup) {
      if (i0 > k) break;
#pragma unroll
      for (int r = 0; r < kRowGroup; ++r) {
        if (i0 + r >= kMaxRows) break;
        ArgMax best{-INFINITY, -1};
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
          const int v = v0 + j * kThreads + threadIdx.x;
          if (v < v1 && (best.i < 0 || x[i0 + r][j] > best.v)) best = ArgMax{x[i0 + r][j], v};   // v grows with j
        }
#pragma unroll
        for (int m = 32; m > 0; m >>= 1) {
          ArgMax o{__shfl_xor(best.v, m, 64), __shfl_xor(best.i, m, 64)};
          best = better(best, o);
        }
        if (lane == 0) sh.gsm[r][w] = best;
      }
      __syncthreads();
      if (threadIdx.x < kRowGroup && i0 + (int)threadIdx.x <= k) {
        const int r = threadIdx.x;
        ArgMax g = sh.gsm[r][0];
        for (int i = 1; i < kWaves; ++i) g = better(g, sh.gsm[r][i]);
        store_partial(out + (size_t)(i0 + r) * nchunks + chunk, g);
      }
      __syncthreads();
    }
    return;
  }
  const int n = accepted_prefix(a, src, b, &sh.n, sh.drafts);
  const int use_q = n < k ? 1 : 0;
  float pv[kPer], qv[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int v = v0 + j * kThreads + threadIdx.x;
    pv[j] = v < v1 ? src.target(b, n, v) : 0.f;
  }
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int v = v0 + j * kThreads + threadIdx.x;
    qv[j] = (use_q && v < v1) ? src.drafted(b, n, v) : 0.f;
  }
  uint64_t sr = 0, sp = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const uint64_t wp = fixed_weight(pv[j]);
    sp += wp;
    sr += use_q ? fixed_weight(fmaxf(0.0f, pv[j] - qv[j])) : wp;
  }
  sr = wave_sum_u64(sr);
  sp = wave_sum_u64(sp);
  if (lane == 0) {
    sh.wsum[w][0] = sr;
    sh.wsum[w][1] = sp;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t tr = 0, tp = 0;
    for (int i = 0; i < kWaves; ++i) {
      tr += sh.wsum[i][0];
      tp += sh.wsum[i][1];
    }
    uint64_t* out = reinterpret_cast<uint64_t*>(parts) + ((size_t)b * nchunks + chunk) * 2;
    publish(out, tr);
    publish(out + 1, tp);
  }
}

// Block-wide exclusive prefix sum of one uint64 per thread; also returns
// the total.  Uses wave prefix sums and the per-wave totals in `tot`.
__device__ uint64_t block_exclusive_scan(uint64_t x, uint64_t* tot, uint64_t* total) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint64_t inc = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = shfl_up_u64(inc, d);
    if (lane >= d) inc += y;
  }
  if (lane == 63) tot[w] = inc;
  __syncthreads();
  uint64_t before = 0, all = 0;
  for (int i = 0; i < kWaves; ++i) {
    if (i < w) before += tot[i];
    all += tot[i];
  }
  __syncthreads();
  *total = all;
  return before + inc - x;
}

// Phase 2, in the last work-group of sequence b: n and the final token
// from every chunk's partials.
template <typename Src>
__device__ void finish_phase(const AcceptArgs& a, const Src& src, const unsigned char* parts, int nchunks, int b,
                             RuleShared& sh) {
  const int c = threadIdx.x;                   // one thread per chunk (nchunks <= 256)
  const int k = a.k, V = a.V;
  const int32_t* draft = a.draft + (size_t)b * k;
  int n = 0, token = 0;
  if (a.mode == 0) {
    // every row's chunk maxima loaded at once (one thread per chunk), the
    // rows' argmaxes formed kRowGroup rows per barrier, then the longest
    // prefix of drafts equal to them
    const ArgMax* part = reinterpret_cast<const ArgMax*>(parts) + (size_t)b * (k + 1) * nchunks;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (c < k) sh.drafts[c] = draft[c];        // read by every thread after the barriers below
    ArgMax r[kMaxRows];
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i)
      r[i] = (i <= k && c < nchunks) ? load_partial(part + (size_t)i * nchunks + c) : ArgMax{-INFINITY, -1};
#pragma unroll
    for (int i0 = 0; i0 < kMaxRows; i0 += kRowGroup) {
      if (i0 > k) break;
#pragma unroll
      for (int rr = 0; rr < kRowGroup; ++rr) {
        if (i0 + rr >= kMaxRows) break;
        ArgMax x = r[i0 + rr];
#pragma unroll
        for (int m = 32; m > 0; m >>= 1) {
          ArgMax o{__shfl_xor(x.v, m, 64), __shfl_xor(x.i, m, 64)};
          x = better(x, o);
        }
        if (lane == 0) sh.gsm[rr][w] = x;
      }
      __syncthreads();
      if (threadIdx.x < kRowGroup && i0 + (int)threadIdx.x <= k) {
        ArgMax g = sh.gsm[threadIdx.x][0];
        for (int i = 1; i < kWaves; ++i) g = better(g, sh.gsm[threadIdx.x][i]);
        sh.gmax[i0 + threadIdx.x] = g;
      }
      __syncthreads();
    }
    int nn = 0;
    while (nn < k && sh.drafts[nn] == sh.gmax[nn].i) ++nn;
    n = nn;
    token = sh.gmax[nn].i;
  } else {
    uint64_t x_res = 0ull, x_p = 0ull;
    if (c < nchunks) {
      const uint64_t* sums = reinterpret_cast<const uint64_t*>(parts) + (size_t)b * nchunks * 2;
      x_res = load_partial(sums + 2 * c);
      x_p = load_partial(sums + 2 * c + 1);
    }
    n = sh.n;                                  // the chunk phase's tests (same work-group)
    // residual weights, else p-only weights, else argmax
    uint64_t S;
    uint64_t x = x_res;
    uint64_t before = block_exclusive_scan(x, sh.tot, &S);
    int sel = 0;
    if (S == 0) {
      sel = 1;
      x = x_p;
      before = block_exclusive_scan(x, sh.tot, &S);
    }
    if (S == 0) {
      token = block_argmax_range([&](int v) { return src.target(b, n, v); }, 0, V, sh.sm).i;
    } else {
      const int use_q = (sel == 0 && n < k) ? 1 : 0;
      float uf = src.uniform(b, k) * 16777216.0f;   // exact: u is a float32
      uf = fminf(fmaxf(floorf(uf), 0.0f), 16777215.0f);
      const uint64_t av = (uint64_t)uf;
      const uint64_t T = av * (S >> 24) + ((av * (S & 0xffffffull)) >> 24);
      // the chunk whose [before, before + x) range holds T (exactly one)
      if (x != 0 && before <= T && T < before + x) {
        sh.chunk = c;
        sh.before = before;
      }
      if (threadIdx.x == 0) sh.tok = 0x7fffffff;
      __syncthreads();
      // inside the chunk, thread t takes the kPerThread consecutive entries
      // from c0 + t kPerThread, all loaded at once; a block prefix sum of
      // the threads' totals finds the thread whose range holds T, and that
      // thread finds the first entry whose inclusive prefix sum exceeds T
      constexpr int kPerThread = kChunk / kThreads;
      const int c0 = sh.chunk * kChunk, c1 = min(V, c0 + kChunk);
      const int e0 = c0 + threadIdx.x * kPerThread;
      uint64_t wv[kPerThread], mine = 0;
#pragma unroll
      for (int j = 0; j < kPerThread; ++j) {
        wv[j] = e0 + j < c1 ? weight_at(src, b, n, e0 + j, use_q) : 0ull;
        mine += wv[j];
      }
      uint64_t chunk_total;
      const uint64_t pre = sh.before + block_exclusive_scan(mine, sh.tot, &chunk_total);
      if (mine != 0 && pre <= T && T < pre + mine) {
        uint64_t incl = pre;
        int hit = -1;
#pragma unroll
        for (int j = 0; j < kPerThread; ++j) {
          incl += wv[j];
          if (hit < 0 && incl > T) hit = e0 + j;
        }
        sh.tok = hit;                          // found: T < pre + mine
      }
      __syncthreads();
      token = sh.tok;
    }
  }
  int32_t* tok = a.tokens + (size_t)b * (k + 1);
  for (int i = threadIdx.x; i <= k; i += kThreads) tok[i] = i < n ? sh.drafts[i] : (i == n ? token : -1);
  if (threadIdx.x == 0) a.n_accepted[b] = n;
}

// The rule: one work-group per (chunk, sequence), chunks fastest on a 1-D grid.  Every work-group writes its chunk's
// partials, publishes them (release fence) and counts its arrival; the one
// that completes the count of its sequence runs the finish and resets the
// counter.  Work-groups never wait for each other, so the grid always
// drains.
template <typename Src>
__global__ __launch_bounds__(kThreads) void accept_rule(AcceptArgs a, Src src, unsigned* count, unsigned char* parts,
                                                        int nchunks) {
  __shared__ RuleShared sh;
  const int chunk = (int)(blockIdx.x % (unsigned)nchunks), b = (int)(blockIdx.x / (unsigned)nchunks);
  src.prepare(b, sh.rows);
  __syncthreads();
  chunk_phase(a, src, parts, nchunks, chunk, b, sh);
  if (!arrive_last(count + (size_t)b * kCounterStride, (unsigned)nchunks, &sh.last)) return;
  finish_phase(a, src, parts, nchunks, b, sh);
}

// Row statistics of the logits at temperature: one work-group per (4096-entry
// chunk, row), chunks fastest on a 1-D grid,
// with rows b (k+1) + i of the target logits, then B (k+1) + b k + i of the
// draft logits; each work-group writes (max, sum 2^(z s - max)) of its chunk.
// Rows whose start is 16-byte aligned are read with 16-byte loads (4 fp32 or
// 8 bf16 logits per load), others one logit at a time.

__device__ __forceinline__ void load16(const float* p, float* x) {
  const floatx4 v = *reinterpret_cast<const floatx4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = v[e];
}
__device__ __forceinline__ void load16(const uint16_t* p, float* x) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(v[e] << 16);
    x[2 * e + 1] = __uint_as_float(v[e] & 0xffff0000u);
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void logit_stats_chunks(const T* zt, const T* zd, float s, int B,
                                                               int k, int V, float2* part, int nchunks) {
  constexpr int PER = 16 / sizeof(T);                    // logits per 16-byte load
  constexpr int NX = kStatChunk / kThreads;              // logits per thread
  __shared__ float2 sm[kWaves];
  const int chunk = (int)(blockIdx.x % (unsigned)nchunks), r = (int)(blockIdx.x / (unsigned)nchunks);
  const int rt = B * (k + 1);
  const T* row = r < rt ? zt + (size_t)r * V : zd + (size_t)(r - rt) * V;
  const int v0 = chunk * kStatChunk, v1 = min(V, v0 + kStatChunk);
  float x[NX];
  if ((reinterpret_cast<uintptr_t>(row) & 15) == 0 && v1 - v0 == kStatChunk) {
#pragma unroll
    for (int j = 0; j < NX / PER; ++j) load16(row + v0 + (j * kThreads + threadIdx.x) * PER, x + j * PER);
  } else {
#pragma unroll
    for (int j = 0; j < NX / PER; ++j)
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int v = v0 + (j * kThreads + threadIdx.x) * PER + e;
        x[j * PER + e] = v < v1 ? load_logit(row, v) : -INFINITY;
      }
  }
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < NX; ++j) {
    x[j] *= s;
    m = fmaxf(m, x[j]);
  }
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if (lane == 0) sm[w].x = m;
  __syncthreads();
  float M = sm[0].x;
  for (int i = 1; i < kWaves; ++i) M = fmaxf(M, sm[i].x);
  float l = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int j = 0; j < NX; ++j) l += fast_exp2(x[j] - M);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
  if (lane == 0) sm[w].y = l;
  __syncthreads();
  if (threadIdx.x == 0) {
    float L = 0.f;
    for (int i = 0; i < kWaves; ++i) L += sm[i].y;
    part[(size_t)r * nchunks + chunk] = make_float2(M, L);
  }
}

__global__ __launch_bounds__(kThreads) void philox_uniforms_kernel(uint64_t seed, uint64_t offset, float* u,
                                                                   int B, int n) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t < B * n) u[t] = philox_uniform(seed, offset, t / n, t % n);
}

template <typename Src>
hipError_t launch_rule(const AcceptArgs& a, const Src& src, unsigned* count, unsigned char* parts, hipStream_t st) {
  const int nchunks = (a.V + kChunk - 1) / kChunk;
  hipLaunchKernelGGL((accept_rule<Src>), dim3(nchunks * a.B), dim3(kThreads), 0, st, a, src, count, parts, nchunks);
  return hipGetLastError();
}

template <typename Src>
hipError_t launch_rule(const AcceptArgs& a, const Src& src, void* ws, hipStream_t st) {
  unsigned char* base = static_cast<unsigned char*>(ws);
  return launch_rule(a, src, reinterpret_cast<unsigned*>(base), base + counter_bytes(a.B), st);
}

template <typename T>
hipError_t launch_logits(const AcceptLogitsArgs& la, void* ws, hipStream_t st) {
  const AcceptArgs& a = la.rule;
  const int nchunks = (a.V + kStatChunk - 1) / kStatChunk;
  const int nrows = a.B * (2 * a.k + 1);
  LogitSrc<T> src{static_cast<const T*>(la.target_logits), static_cast<const T*>(la.draft_logits), nullptr,
                  nchunks, nullptr, la.scale_log2, la.seed, la.offset, a.B, a.k, a.V};
  unsigned char* base = static_cast<unsigned char*>(ws);
  if (a.mode != 0) {
    float2* part = reinterpret_cast<float2*>(base);
    hipLaunchKernelGGL((logit_stats_chunks<T>), dim3(nchunks * nrows), dim3(kThreads), 0, st, src.zt, src.zd,
                       la.scale_log2, a.B, a.k, a.V, part, nchunks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    src.part = part;
    base += ((size_t)nrows * nchunks * sizeof(float2) + 255) / 256 * 256;
  }
  return launch_rule(a, src, base, st);
}

}  // namespace

size_t accept_logits_workspace_bytes(int B, int k, int V, int mode) {
  const int nchunks = (V + kStatChunk - 1) / kStatChunk;
  size_t stats = 0;
  if (mode != 0) stats = ((size_t)B * (2 * k + 1) * nchunks * sizeof(float2) + 255) / 256 * 256;
  return stats + accept_workspace_bytes(B, k, V, mode);
}

hipError_t launch_accept_logits(const AcceptLogitsArgs& la, int dtype, void* ws, hipStream_t st) {
  return dtype == 0 ? launch_logits<float>(la, ws, st) : launch_logits<uint16_t>(la, ws, st);
}

hipError_t launch_philox_uniforms(uint64_t seed, uint64_t offset, float* u, int B, int n, hipStream_t st) {
  const long long total = (long long)B * n;
  hipLaunchKernelGGL(philox_uniforms_kernel, dim3((unsigned)((total + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     st, seed, offset, u, B, n);
  return hipGetLastError();
}

size_t accept_workspace_bytes(int B, int k, int V, int mode) {
  const int nchunks = (V + kChunk - 1) / kChunk;
  if (mode == 0) return counter_bytes(B) + (size_t)B * (k + 1) * nchunks * sizeof(ArgMax);
  return counter_bytes(B) + (size_t)B * nchunks * 2 * sizeof(uint64_t);
}

hipError_t launch_accept(const AcceptArgs& a, void* ws, hipStream_t st) {
  return launch_rule(a, ProbSrc{a.p, a.q, a.u, a.k, a.V}, ws, st);
}

size_t accept_partial_bytes(int B, int k, int V, int mode) {
  return accept_workspace_bytes(B, k, V, mode) - counter_bytes(B);
}

hipError_t launch_accept_split(const AcceptArgs& a, unsigned* counters, void* partials, hipStream_t st) {
  return launch_rule(a, ProbSrc{a.p, a.q, a.u, a.k, a.V}, counters, static_cast<unsigned char*>(partials), st);
}

}  // namespace sd
