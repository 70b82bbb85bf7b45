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

constexpr int kTile = 32;       // keys per wave iteration
constexpr int kWaves = 4;       // waves per work-group
constexpr int kVPad = 8;        // bf16 padding per LDS row of the V tile

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short shortx4;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

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
template <int D, int RB, bool PAGED>
__global__ __launch_bounds__(256) void verify_split_bf16(VerifyArgs a, int keys_per_split,
                                                         int nsplit, int row_groups,
                                                         int rows_padded) {
  constexpr int DC = D / 32;              // 32-channel K slices (QK^T)
  constexpr int DB = D / 16;              // 16-channel output blocks (PV)
  constexpr int PK = D / 8;               // 16-byte pieces per key row
  constexpr int VSTR = D + kVPad;         // LDS row stride of V (elements)
  constexpr int NV = kTile * PK / kWave;  // V pieces per lane per tile
  extern __shared__ __align__(16) unsigned char smem[];

  const int split = blockIdx.x;
  const int hk = blockIdx.y / row_groups;
  const int rg = blockIdx.y % row_groups;
  const int b = blockIdx.z;
  const int L = seq_len(a, b, PAGED);
  const int k0 = split * keys_per_split;
  if (k0 >= L) return;                    // the merge skips empty splits
  const int k1 = min(L, k0 + keys_per_split);

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, G = lane >> 4, c = lane & 15;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int row0 = rg * RB * 16;

  // This lane's query rows: row row0 + rb*16 + c, block position j = row / g,
  // query head hk * g + row % g.  B operand of S^T = K Q^T.
  bf16x8 qf[RB][DC];
  int lim[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = row0 + rb * 16 + c;
    if (r < R) {
      const int j = r / g;
      const int h = hk * g + (r - j * g);
      const uint4* src = reinterpret_cast<const uint4*>(
          static_cast<const uint16_t*>(a.q) + (((size_t)b * a.k + j) * a.Hq + h) * D);
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = src[dc * 4 + G];
        qf[rb][dc] = pk.b;
      }
      lim[rb] = L - a.k + j;              // last visible key of this row
    } else {
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = make_uint4(0, 0, 0, 0);
        qf[rb][dc] = pk.b;
      }
      lim[rb] = -1;
    }
  }

  float m[RB], l[RB];
  floatx4 o[RB][DB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  uint16_t* vs = reinterpret_cast<uint16_t*>(smem) + w * kTile * VSTR;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.kc);
  const uint16_t* vbase = static_cast<const uint16_t*>(a.vc);
  const int ntiles = (k1 - k0 + kTile - 1) / kTile;

  // register prefetch of one tile ahead
  uint4 kn[2][DC];
  uint4 vn[NV];
  auto load_tile = [&](int tile) {
    const int t0 = k0 + tile * kTile;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int t = min(t0 + kb * 16 + c, L - 1);
      const uint4* src = reinterpret_cast<const uint4*>(kbase + kv_offset<PAGED>(a, b, hk, t, D));
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) kn[kb][dc] = src[dc * 4 + G];
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int p = lane + kWave * i;
      const int t = min(t0 + p / PK, L - 1);
      vn[i] = reinterpret_cast<const uint4*>(vbase + kv_offset<PAGED>(a, b, hk, t, D))[p % PK];
    }
  };

  if (w < ntiles) load_tile(w);
  for (int tile = w; tile < ntiles; tile += kWaves) {
    const int t0 = k0 + tile * kTile;
    bf16x8 kf[2][DC];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        Pack8 pk;
        pk.u = kn[kb][dc];
        kf[kb][dc] = pk.b;
      }
    // stage V in this wave's LDS slice, row-major [key][channel]
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int p = lane + kWave * i;
      *reinterpret_cast<uint4*>(vs + (p / PK) * VSTR + (p % PK) * 8) = vn[i];
    }
    if (tile + kWaves < ntiles) load_tile(tile + kWaves);

    // S^T = K Q^T: lane holds S[row rb*16 + c][key t0 + kb*16 + 4G + i]
    floatx4 s[2][RB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dc = 0; dc < DC; ++dc) acc = mfma_bf16(kf[kb][dc], qf[rb][dc], acc);
        s[kb][rb] = acc;
      }

    // online softmax, one row per lane and row block
    bf16x8 ph[RB], pl[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float x[8];
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + kb * 16 + 4 * G + i;
          const float v = (t <= lim[rb]) ? s[kb][rb][i] * a.scale_log2 : -INFINITY;
          x[kb * 4 + i] = v;
          tmax = fmaxf(tmax, v);
        }
      tmax = wave_max_across_groups(tmax);
      const float mnew = fmaxf(m[rb], tmax);
      float alpha = 1.f;
      if (mnew == -INFINITY) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = 0.f;
      } else {
        alpha = exp2f(m[rb] - mnew);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = exp2f(x[e] - mnew);
      }
      m[rb] = mnew;
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) psum += x[e];
      l[rb] = l[rb] * alpha + psum;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const __bf16 hi = float_to_bf16(x[e]);
        ph[rb][e] = hi;
        pl[rb][e] = float_to_bf16(x[e] - bf16_to_float(hi));
      }
    }

    // LDS writes of this wave must land before its lanes read them back
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // O^T += V^T P^T.  K index of the product = keys {4G..4G+3, 16+4G..16+4G+3},
    // the same order in which the accumulator handed this lane its P values.
    // ds_read_tr16_b64: lane j of group G addresses key 4G + j/4 (+16) at
    // channels db*16 + 4*(j%4); lane c then receives 4 keys at channel db*16 + c.
    const int key_a = 4 * G + (c >> 2);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int ch = db * 16 + 4 * (c & 3);
      const shortx4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_shortx4*)((__attribute__((address_space(3))) uint16_t*)(vs + key_a * VSTR + ch)));
      const shortx4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_shortx4*)((__attribute__((address_space(3))) uint16_t*)(vs + (key_a + 16) * VSTR + ch)));
      Pack8 vt;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vt.s[e] = (uint16_t)v0[e];
        vt.s[4 + e] = (uint16_t)v1[e];
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        o[rb][db] = mfma_bf16(vt.b, ph[rb], o[rb][db]);
        o[rb][db] = mfma_bf16(vt.b, pl[rb], o[rb][db]);
      }
    }
  }

  // ---- merge the 4 waves of this work-group (fixed order, no atomics)
  float* sm = reinterpret_cast<float*>(smem);
  float* sm_m = sm;                        // [4][RB*16]
  float* sm_l = sm + kWaves * RB * 16;     // [4][RB*16]
  float* ob = sm + 2 * kWaves * RB * 16;   // [RB*16][D + 4]
  constexpr int OSTR = D + 4;
  __syncthreads();                         // all waves are done with V tiles
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    l[rb] = wave_sum_across_groups(l[rb]);
    if (G == 0) {
      sm_m[w * RB * 16 + rb * 16 + c] = m[rb];
      sm_l[w * RB * 16 + rb * 16 + c] = l[rb];
    }
  }
  __syncthreads();
  float ltot[RB], mtot[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    float mx = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) mx = fmaxf(mx, sm_m[ww * RB * 16 + rb * 16 + c]);
    float lt = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww)
        lt += sm_l[ww * RB * 16 + rb * 16 + c] * exp2f(sm_m[ww * RB * 16 + rb * 16 + c] - mx);
    }
    const float f = (mx == -INFINITY) ? 0.f : exp2f(m[rb] - mx);
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] *= f;
    mtot[rb] = mx;
    ltot[rb] = lt;
  }
  auto store_o = [&]() {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<floatx4*>(ob + (rb * 16 + c) * OSTR + db * 16 + 4 * G) = o[rb][db];
  };
  auto add_o = [&]() {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        o[rb][db] += *reinterpret_cast<const floatx4*>(ob + (rb * 16 + c) * OSTR + db * 16 + 4 * G);
  };
  // one staging buffer, fixed order: (O0 + O1) + (O2 + O3)
  if (w == 1) store_o();
  __syncthreads();
  if (w == 0) add_o();
  __syncthreads();
  if (w == 3) store_o();
  __syncthreads();
  if (w == 2) add_o();
  __syncthreads();
  if (w == 2) store_o();
  __syncthreads();
  if (w == 0) {
    add_o();
    const size_t base = ((size_t)(b * a.Hkv + hk) * nsplit + split) * rows_padded + row0;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float inv = ltot[rb] > 0.f ? 1.f / ltot[rb] : 0.f;
      float* dst = a.part_o + (base + rb * 16 + c) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        floatx4 v = o[rb][db] * inv;
        *reinterpret_cast<floatx4*>(dst + db * 16 + 4 * G) = v;
      }
      if (G == 0)
        a.part_lse[base + rb * 16 + c] =
            ltot[rb] > 0.f ? mtot[rb] + log2f(ltot[rb]) : -INFINITY;
    }
  }
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
// One work-group per (sequence, KV head); threads over (row, 4 channels).
__global__ __launch_bounds__(256) void verify_merge(VerifyArgs a, int keys_per_split,
                                                    int nsplit, int rows_padded, int paged) {
  const int hk = blockIdx.x;
  const int b = blockIdx.y;
  const int D = a.D;
  const int g = a.Hq / a.Hkv;
  const int R = a.k * g;
  const int L = seq_len(a, b, paged != 0);
  const int nvalid = min(nsplit, (L + keys_per_split - 1) / keys_per_split);
  const size_t base = (size_t)(b * a.Hkv + hk) * nsplit * rows_padded;
  const int D4 = D / 4;
  for (int i = threadIdx.x; i < R * D4; i += blockDim.x) {
    const int r = i / D4, d4 = i % D4;
    float mx = -INFINITY;
    for (int s = 0; s < nvalid; ++s) mx = fmaxf(mx, a.part_lse[base + (size_t)s * rows_padded + r]);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    if (mx != -INFINITY) {
      for (int s = 0; s < nvalid; ++s) {
        const size_t pr = base + (size_t)s * rows_padded + r;
        const float ls = a.part_lse[pr];
        if (ls == -INFINITY) continue;
        const float wgt = exp2f(ls - mx);
        wsum += wgt;
        acc += wgt * *reinterpret_cast<const floatx4*>(a.part_o + pr * D + d4 * 4);
      }
    }
    const int j = r / g;
    const int h = hk * g + (r - j * g);
    const size_t orow = ((size_t)b * a.k + j) * a.Hq + h;
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    *reinterpret_cast<floatx4*>(a.out + orow * D + d4 * 4) = acc * inv;
    if (a.lse != nullptr && d4 == 0)
      a.lse[orow] = wsum > 0.f ? (mx + log2f(wsum)) * kLn2 : -INFINITY;
  }
}

template <int D, int RB, bool PAGED>
hipError_t launch_bf16(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  constexpr int VSTR = D + kVPad;
  const size_t v_bytes = (size_t)kWaves * kTile * VSTR * 2;
  const size_t m_bytes = (size_t)(2 * kWaves * RB * 16 + RB * 16 * (D + 4)) * 4;
  const size_t lds = std::max(v_bytes, m_bytes);
  dim3 grid(p.nsplit, a.Hkv * p.row_groups, a.B);
  hipLaunchKernelGGL((verify_split_bf16<D, RB, PAGED>), grid, dim3(256), lds, st, a,
                     p.keys_per_split, p.nsplit, p.row_groups, p.rows_padded);
  return hipGetLastError();
}

template <int D, bool PAGED>
hipError_t dispatch_rb(const VerifyArgs& a, const VerifyPlan& p, hipStream_t st) {
  switch (p.row_blocks) {
    case 1: return launch_bf16<D, 1, PAGED>(a, p, st);
    case 2: return launch_bf16<D, 2, PAGED>(a, p, st);
    case 3: return launch_bf16<D, 3, PAGED>(a, p, st);
    default: return launch_bf16<D, 4, PAGED>(a, p, st);
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
    p.row_blocks = std::min(4, blocks16);
    p.row_groups = (blocks16 + p.row_blocks - 1) / p.row_blocks;
    p.rows_padded = p.row_groups * p.row_blocks * 16;
    // Enough work-groups to fill 256 compute units about twice, with at
    // least 128 keys (one tile per wave) per split.
    const long long pairs = (long long)B * Hkv * p.row_groups;
    const long long target = 512;
    long long nsplit = std::max(1LL, (target + pairs - 1) / pairs);
    long long kps = (capacity + nsplit - 1) / nsplit;
    kps = std::max(128LL, (kps + 127) / 128 * 128);
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
  hipLaunchKernelGGL(verify_merge, dim3(a.Hkv, a.B), dim3(256), 0, st, a, p.keys_per_split,
                     p.nsplit, p.rows_padded, paged ? 1 : 0);
  return hipGetLastError();
}

}  // namespace sd
