// Device helpers shared by the gfx950 kernels: vector types, matrix-core
// wrappers, bf16 / fp16 conversions and wavefront reductions.
//
// Matrix-core lane layout used throughout (64-lane wavefront, lane l,
// group G = l / 16, column c = l % 16), for D[16x16] += A[16xK] * B[Kx16]:
//   A operand: lane l holds A[c][K-slice of group G]
//   B operand: lane l holds B[K-slice of group G][c]
//   accumulator: lane l holds D[4G + i][c], i = 0..3
// Any assignment of the K index to (G, element) is valid as long as A and B
// use the same one; the kernels exploit that freedom to read contiguous
// memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;
// 16 raw bytes as a native vector (HIP's uint4 is a class that register
// promotion of arrays does not always see through)
typedef __attribute__((__vector_size__(4 * sizeof(unsigned)))) unsigned u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(unsigned)))) unsigned u32x2;

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ floatx4 mfma_bf16(const bf16x8& a, const bf16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f16(const f16x8& a, const f16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f32(float a, float b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// bf16 bit pattern <-> float (exact widening; narrowing rounds to nearest even)
__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ __bf16 float_to_bf16(float x) {
  return (__bf16)x;   // round to nearest even
}

__device__ __forceinline__ float bf16_to_float(__bf16 x) {
  return (float)x;
}

// 2^x with the hardware instruction (inputs far below -126 give 0)
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte vector of 8 bf16 values viewed as raw words
union Pack8 {
  u32x4 u;
  bf16x8 b;
  f16x8 h;
  uint16_t s[8];
};

// LDS reads issued as inline asm.  The compiler does not see them as LDS
// loads, so it never holds them back behind LDS-DMA copies it cannot prove
// disjoint; the caller orders them with lds_wait() + tie() instead.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) void*)p);
}

__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

// same, with a compile-time byte offset folded into the instruction
template <int OFF>
__device__ __forceinline__ u32x4 lds_read_b128_off(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr16_b64_off(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

__device__ __forceinline__ u32x2 lds_read_b64(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

// 8-byte transposing read: within each 16-lane group, lane i receives
// element i % 4 of the 8-byte blocks addressed by lanes i/4, i/4 + 4,
// i/4 + 8 and i/4 + 12 of that group.
__device__ __forceinline__ u32x2 lds_read_tr16_b64(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

// one signed byte, sign-extended
__device__ __forceinline__ int lds_read_i8(uint32_t addr) {
  int r;
  asm volatile("ds_read_i8 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

__device__ __forceinline__ void lds_write_b128(uint32_t addr, const u32x4& v) {
  asm volatile("ds_write_b128 %0, %1" : : "v"(addr), "v"(v));
}

template <int OFF>
__device__ __forceinline__ void lds_write_b128_off(uint32_t addr, const u32x4& v) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_write_b128 %0, %1 offset:%2" : : "v"(addr), "v"(v), "i"(OFF));
}

// Wait for every LDS operation of this wave (asm reads included).
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Wait until at most N of this wave's LDS operations are outstanding.  LDS
// operations complete in issue order, so with the N most recent ones still
// in flight every earlier one has finished (counts above the counter's
// 4-bit range wait for 15, which is stricter).
template <int N>
__device__ __forceinline__ void lds_wait_n() {
  static_assert(N >= 0, "count");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N < 15 ? N : 15) : "memory");
}

// Make a register value depend on the preceding volatile asm (the wait), so
// no use of it can be scheduled before the wait.
template <typename T>
__device__ __forceinline__ void tie(T& x) {
  asm volatile("" : "+v"(x));
}

// LDS swizzle of the 16-byte pieces of tile row t (a token or key) for rows
// of PK pieces: piece p is stored at slot p ^ lds_swizzle<PK>(t).  gfx950's
// LDS has 64 four-byte banks.  The 8-byte transposing read serves 32 lanes
// per pass, so 8 consecutive rows read at two adjacent pieces each
// (transposed fragments of 4 rows x 4 elements per 16 lanes) must fill the
// 256 bank bytes.  The 16-byte read serves 16 lanes per pass, but the pass
// pairs lanes 0..7 of one group of 16 with lanes 8..15 of the neighbouring
// group (measured with the bank-conflict counter: matrix-core fragments of
// 16 rows x 8 elements, lane 16 G + c reading row c at piece 4 dc + G, go
// 2-way conflicted when rows c and c + 8 take slots that differ in bit 0,
// conflict-free when the swizzle leaves bit 0 alone).
// For 256-byte rows (PK = 16) the swizzle is (t & 7) << 1: bits 1..3 differ
// within each aligned 8 rows and bit 0 never moves; for 128-byte rows (PK =
// 8, two rows per bank row) a permutation of 0..7 on each row parity whose
// bits 1..2 differ within each aligned quad of that parity.
template <int PK>
__device__ __forceinline__ constexpr int lds_swizzle(int t) {
  static_assert(PK == 8 || PK == 16, "rows of 128 or 256 bytes");
  t &= 15;
  if constexpr (PK == 16) {
    return (t & 7) << 1;
  } else {
    const int u = (t >> 1) & 7;
    return ((u & 3) << 1) | (u >> 2);
  }
}

// Reductions over the four lanes l, l^16, l^32, l^48 (same column c, the
// four groups).  gfx950's v_permlane32_swap / v_permlane16_swap exchange
// halves / odd-even rows of two registers; applied to two copies of v they
// hand every lane its partner's value without an LDS round trip.
// Wait until at most N vector-memory operations of this wave are in flight
// (and all of its LDS operations are done), then meet the other waves.  The
// empty asm statements keep the compiler from moving memory accesses across
// the barrier; the barrier itself carries no fence, because a fence would
// wait for every LDS DMA in flight (including the tiles being prefetched).
template <int N>
__device__ __forceinline__ void wait_vm_then_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Hand-off between work-groups of one launch (the last of a group of
// work-groups to finish combines their partial results).  Partials are
// written with device-scope stores, which write through to the level that
// every XCD shares, and read back with device-scope loads, so neither side
// needs a cache write-back or invalidate (an agent-scope fence costs both,
// over the whole L2, in every work-group).  arrive_last() waits until this
// wave's stores have completed, meets the work-group, counts its arrival
// with a device-scope atomic and tells every thread whether it was the last
// of `expected`; the last one resets the counter to zero for the next use.
// No work-group ever waits for another, so the grid always drains.
__device__ __forceinline__ void publish(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void publish(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t fetch_published(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float fetch_published(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool arrive_last(unsigned* counter, unsigned expected, int* lds_flag) {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));    // vmcnt(0): this wave's stores are done
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = prev + 1u == expected;
    if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *lds_flag = last;
  }
  __syncthreads();
  return *lds_flag != 0;
}

// Stage rows 0 .. nrows-1 of ncols elements (row r of source k at
// src[k] + row_off(r), aligned to 4 NWORD bytes; ncols a multiple of the
// elements per load) into LDS as floats, dst[k][r * DS + c] (bf16 widened
// exactly), with loads of NWORD 32-bit words (4: 16 bytes), NB per thread
// and source in flight: every load of a batch is issued before any of its
// values is stored, so a batch costs one memory latency instead of one
// per element.  NS sources share the rows.
template <int NB, int NS, int NWORD, typename T, typename RowOff>
__device__ __forceinline__ void stage_rows(float* const (&dst)[NS], int DS, const T* const (&src)[NS],
                                           RowOff row_off, int nrows, int ncols) {
  static_assert(NWORD == 1 || NWORD == 4, "4- or 16-byte loads");
  typedef __attribute__((__vector_size__(NWORD * sizeof(uint32_t)))) uint32_t words;
  constexpr int PER = (int)sizeof(uint32_t) / (int)sizeof(T);   // elements per word
  constexpr int V = NWORD * PER;                                 // elements per load
  const int per_row = ncols / V;
  const int total = nrows * per_row;
  for (int base = threadIdx.x; base < total; base += NB * (int)blockDim.x) {
    words v[NS][NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int i = base + j * (int)blockDim.x;
      if (i < total) {
        const int r = i / per_row;
        const size_t off = row_off(r) + (size_t)(i - r * per_row) * V;
#pragma unroll
        for (int k = 0; k < NS; ++k) v[k][j] = *reinterpret_cast<const words*>(src[k] + off);
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int i = base + j * (int)blockDim.x;
      if (i < total) {
        const int r = i / per_row, c = (i - r * per_row) * V;
#pragma unroll
        for (int k = 0; k < NS; ++k) {
          float* d = dst[k] + r * DS + c;
#pragma unroll
          for (int e = 0; e < NWORD; ++e) {
            const uint32_t x = v[k][j][e];
            if constexpr (PER == 1) {
              d[e] = __uint_as_float(x);
            } else {
              d[2 * e] = __uint_as_float(x << 16);
              d[2 * e + 1] = __uint_as_float(x & 0xffff0000u);
            }
          }
        }
      }
    }
  }
}

// two bf16 -> two fp16, rounded to nearest even: exact for zero and every
// magnitude in 2^-17 .. 65280 (all bf16 values there fit fp16's 11-bit
// significand); larger magnitudes become +-inf, which the callers detect.
typedef _Float16 half2_ __attribute__((ext_vector_type(2)));
typedef float float2_ __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t v) {
  const float lo = __uint_as_float(v << 16);
  const float hi = __uint_as_float(v & 0xffff0000u);
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2_){lo, hi}, half2_));
}

// 16 int8 values q (one 16-byte piece) to 16 fp16 values q * 2^e, exact
// for e in [-14, 9] (|q| <= 127: every result is zero or a normal fp16).
// Per 4 values: the bytes biased to u = q + 128, placed under the fp16
// pattern of 1024 (0x64uu = 1024 + u) by byte permutes, then 1152
// subtracted and 2^e applied with packed fp16 arithmetic (both exact).
__device__ __forceinline__ void i8x16_to_f16_pow2(const u32x4& q, int e, u32x4& lo, u32x4& hi) {
  const uint32_t s_bits = (uint32_t)(e + 15) << 10;          // 2^e as fp16
  const half2_ s2 = __builtin_bit_cast(half2_, s_bits | (s_bits << 16));
  const half2_ off = {(_Float16)-1152.f, (_Float16)-1152.f};
  uint32_t r[8];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t u = q[k] ^ 0x80808080u;
    const uint32_t p01 = __builtin_amdgcn_perm(0x64646464u, u, 0x04010400u);   // 0x64 u1 0x64 u0
    const uint32_t p23 = __builtin_amdgcn_perm(0x64646464u, u, 0x04030402u);   // 0x64 u3 0x64 u2
    r[2 * k] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(half2_, p01) + off) * s2);
    r[2 * k + 1] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(half2_, p23) + off) * s2);
  }
  lo = u32x4{r[0], r[1], r[2], r[3]};
  hi = u32x4{r[4], r[5], r[6], r[7]};
}

__device__ __forceinline__ float partner32(float v, float* other) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  *other = __uint_as_float(r[1]);
  return __uint_as_float(r[0]);
}

__device__ __forceinline__ float partner16(float v, float* other) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  *other = __uint_as_float(r[1]);
  return __uint_as_float(r[0]);
}

__device__ __forceinline__ float wave_max_across_groups(float v) {
  float o;
  float a = partner32(v, &o);
  v = fmaxf(a, o);
  a = partner16(v, &o);
  return fmaxf(a, o);
}

__device__ __forceinline__ float wave_sum_across_groups(float v) {
  float o;
  float a = partner32(v, &o);
  v = a + o;
  a = partner16(v, &o);
  return a + o;
}

}  // namespace sd
