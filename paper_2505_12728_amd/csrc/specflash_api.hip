// C ABI entry points: host-side validation, planning and launch.  Nothing is
// enqueued unless every argument check passes; the library allocates no
// device memory.  Its only state is the per-device cache of compute-unit
// counts below (written once per device with the value the runtime reports).
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "../../include/specflash.h"
#include "launch.hpp"

namespace {

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

int status_from(hipError_t e) { return e == hipSuccess ? SD_OK : SD_ERR_HIP; }

bool verify_shape_ok(int B, int k, int Hq, int Hkv, int D, int dtype, int* status) {
  if (B < 1 || k < 1 || Hq < 1 || Hkv < 1 || (dtype != SD_F32 && dtype != SD_BF16)) {
    *status = SD_ERR_INVALID_ARG;
    return false;
  }
  if (Hq % Hkv != 0) {
    *status = SD_ERR_INVALID_ARG;
    return false;
  }
  const int rows = k * (Hq / Hkv);
  if (k > 16 || (D != 64 && D != 128) || rows > 256 || (dtype == SD_F32 && rows > 64)) {
    *status = SD_ERR_UNSUPPORTED;
    return false;
  }
  return true;
}

bool compress_shape_ok(int B, int N, int C, int d, int H, int dtype, int* status) {
  if (B < 1 || N < 1 || C < 1 || d < 1 || H < 1 || d % H != 0 ||
      (dtype != SD_F32 && dtype != SD_BF16)) {
    *status = SD_ERR_INVALID_ARG;
    return false;
  }
  const int dh = d / H;
  const bool ok = dh == 64 || dh == 128 || dh == 256;
  if (!ok || N > (1 << 24) || C > (1 << 20) || d > (1 << 22)) {
    *status = SD_ERR_UNSUPPORTED;
    return false;
  }
  return true;
}

}  // namespace

// ------------------------------------------- scratch of the allocation-free entry point
// sd_spec_accept_noalloc keeps its counters and partials in `scratch`, a
// device array of fixed size: arrival counters of up to kScratchSeqs
// sequences at offset 0 (their place never depends on the call's shape),
// then the chunk partials.  Host code never uses the array's name as an
// address: its device address comes from hipGetSymbolAddress, once per
// device, and every use (kernel arguments, the clearing kernel) goes
// through that pointer.
namespace {
constexpr size_t kScratchBytes = size_t(4) << 20;      // 4 MiB per device
constexpr int kScratchSeqs = 1024;
constexpr int kScratchCounterWords = kScratchSeqs * sd::kCounterStride;
constexpr size_t kScratchCounterBytes = (size_t)kScratchCounterWords * sizeof(unsigned);
static_assert(kScratchCounterBytes % 256 == 0, "partials start 256-byte aligned");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

__global__ void zero_words(unsigned* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

struct ScratchSlot {
  std::once_flag once;
  unsigned char* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[64];

// Device address of this device's scratch (set-up on its first use: the
// address is looked up with the device current and the counters are
// cleared on `st`, ahead of any kernel that reads them).
hipError_t scratch_for_current_device(hipStream_t st, unsigned char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&] {
    void* p = nullptr;
    slot.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (slot.err != hipSuccess) return;
    hipLaunchKernelGGL(zero_words, dim3((kScratchCounterWords + 255) / 256), dim3(256), 0, st,
                       static_cast<unsigned*>(p), kScratchCounterWords);
    slot.err = hipGetLastError();
    if (slot.err == hipSuccess) slot.ptr = static_cast<unsigned char*>(p);
  });
  *out = slot.ptr;
  return slot.err;
}
}  // namespace

extern "C" {

const char* sd_status_string(int status) {
  switch (status) {
    case SD_OK: return "SD_OK";
    case SD_ERR_INVALID_ARG: return "SD_ERR_INVALID_ARG: invalid argument";
    case SD_ERR_UNSUPPORTED: return "SD_ERR_UNSUPPORTED: shape or dtype not supported";
    case SD_ERR_WORKSPACE: return "SD_ERR_WORKSPACE: workspace missing or too small";
    case SD_ERR_HIP: return "SD_ERR_HIP: HIP runtime error at launch";
    default: return "unknown sd_status";
  }
}

int sd_version(void) { return (1 << 16) | 0; }

// Compute units of the current device (cached per device; 256 when no
// device can be queried, e.g. for sizing on a host without a GPU).  Every
// writer stores the same value, and the atomics make concurrent first calls
// from several host threads well defined.
static int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    const int c = cached[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return 256;
  if (dev < 64) cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

// ------------------------------------------------------------- compress
size_t sd_latent_compress_workspace_size(int B, int N, int C, int d, int num_heads, int dtype) {
  int st;
  if (!compress_shape_ok(B, N, C, d, num_heads, dtype, &st)) return 0;
  return sd::plan_compress(B, N, C, d, num_heads, dtype, device_cus()).workspace_bytes;
}

int sd_latent_compress(const void* latents, const void* feats, float* out, int B, int N, int C,
                       int d, int num_heads, float scale, int dtype, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = SD_OK;
  if (!compress_shape_ok(B, N, C, d, num_heads, dtype, &st)) return st;
  if (!latents || !feats || !out || !isfinite(scale)) return SD_ERR_INVALID_ARG;
  if (!aligned(latents, 16) || !aligned(feats, 16) || !aligned(out, 16)) return SD_ERR_INVALID_ARG;
  const sd::CompressPlan plan = sd::plan_compress(B, N, C, d, num_heads, dtype, device_cus());
  if (plan.workspace_bytes > 0 && (!workspace || workspace_bytes < plan.workspace_bytes ||
                                   !aligned(workspace, 16)))
    return SD_ERR_WORKSPACE;
  sd::CompressArgs a{};
  a.latents = latents;
  a.feats = feats;
  a.out = out;
  a.B = B;
  a.N = N;
  a.C = C;
  a.d = d;
  a.H = num_heads;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  if (plan.workspace_bytes > 0) {
    a.part_o = static_cast<float*>(workspace);
    a.part_lse = a.part_o + (size_t)B * num_heads * plan.nsplit * C * plan.dh;
  }
  return status_from(sd::launch_compress(a, plan, dtype, static_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------ compress (int8)
size_t sd_latent_compress_q8_workspace_size(int B, int N, int C, int d, int num_heads) {
  int st = SD_OK;
  if (!compress_shape_ok(B, N, C, d, num_heads, SD_BF16, &st) || d / num_heads != 128) return 0;
  return sd::plan_compress(B, N, C, d, num_heads, sd::kCompressInt8, device_cus()).workspace_bytes;
}

int sd_latent_compress_q8(const int8_t* latents_q, const int8_t* latent_exp, const int8_t* feats_q,
                          const int8_t* feat_exp, float* out, int B, int N, int C, int d, int num_heads,
                          float scale, void* workspace, size_t workspace_bytes, void* stream) {
  int st = SD_OK;
  if (!compress_shape_ok(B, N, C, d, num_heads, SD_BF16, &st)) return st;
  if (d / num_heads != 128) return SD_ERR_UNSUPPORTED;
  if (!latents_q || !latent_exp || !feats_q || !feat_exp || !out || !isfinite(scale))
    return SD_ERR_INVALID_ARG;
  if (!aligned(latents_q, 16) || !aligned(feats_q, 16) || !aligned(out, 16)) return SD_ERR_INVALID_ARG;
  const sd::CompressPlan plan = sd::plan_compress(B, N, C, d, num_heads, sd::kCompressInt8, device_cus());
  if (plan.workspace_bytes > 0 && (!workspace || workspace_bytes < plan.workspace_bytes ||
                                   !aligned(workspace, 16)))
    return SD_ERR_WORKSPACE;
  sd::CompressArgs a{};
  a.latents = latents_q;
  a.feats = feats_q;
  a.latent_exp = latent_exp;
  a.feat_exp = feat_exp;
  a.out = out;
  a.B = B;
  a.N = N;
  a.C = C;
  a.d = d;
  a.H = num_heads;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  if (plan.workspace_bytes > 0) {
    a.part_o = static_cast<float*>(workspace);
    a.part_lse = a.part_o + (size_t)B * num_heads * plan.nsplit * C * plan.dh;
  }
  return status_from(sd::launch_compress(a, plan, sd::kCompressInt8, static_cast<hipStream_t>(stream)));
}

// --------------------------------------------------------------- verify
size_t sd_verify_workspace_size(int B, int k, int Hq, int Hkv, int D, int capacity, int dtype) {
  int st;
  if (!verify_shape_ok(B, k, Hq, Hkv, D, dtype, &st) || capacity < 1) return 0;
  const sd::VerifyPlan plan = sd::plan_verify(B, k, Hq, Hkv, D, capacity, dtype, device_cus());
  return plan.ok ? plan.workspace_bytes : 0;
}

int sd_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* kv_len, const int32_t* page_table, int max_pages,
                        int num_pages, int Lmax, float* out, float* lse, int B, int k, int Hq,
                        int Hkv, int D, float scale, int dtype, void* workspace,
                        size_t workspace_bytes, void* stream) {
  int st = SD_OK;
  if (!verify_shape_ok(B, k, Hq, Hkv, D, dtype, &st)) return st;
  if (!q || !k_cache || !v_cache || !kv_len || !out || !isfinite(scale)) return SD_ERR_INVALID_ARG;
  const size_t al = dtype == SD_BF16 ? 16 : 4;
  if (!aligned(q, al) || !aligned(k_cache, al) || !aligned(v_cache, al) || !aligned(out, 16) ||
      !aligned(kv_len, 4) || (lse && !aligned(lse, 4)))
    return SD_ERR_INVALID_ARG;
  int capacity;
  if (page_table) {
    if (max_pages < 1 || num_pages < 1 || max_pages > (1 << 26) || !aligned(page_table, 4))
      return SD_ERR_INVALID_ARG;
    capacity = max_pages * 16;
  } else {
    if (Lmax < 1) return SD_ERR_INVALID_ARG;
    capacity = Lmax;
  }
  const sd::VerifyPlan plan = sd::plan_verify(B, k, Hq, Hkv, D, capacity, dtype, device_cus());
  if (!plan.ok) return SD_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < plan.workspace_bytes || !aligned(workspace, 16))
    return SD_ERR_WORKSPACE;
  sd::VerifyArgs a{};
  a.q = q;
  a.kc = k_cache;
  a.vc = v_cache;
  a.kv_len = kv_len;
  a.page_table = page_table;
  a.max_pages = max_pages;
  a.num_pages = num_pages;
  a.Lmax = Lmax;
  a.out = out;
  a.lse = lse;
  a.B = B;
  a.k = k;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.part_o = static_cast<float*>(workspace);
  a.part_lse = a.part_o + plan.part_rows * D;
  return status_from(sd::launch_verify(a, plan, dtype, static_cast<hipStream_t>(stream)));
}

// --------------------------------------------------------------- accept
// batch bounds: one work-group per (1024-entry chunk, sequence) and, from
// logits, per (4096-entry chunk, logit row), counted on a 1-D grid below 2^31
constexpr int kAcceptMaxSeqs = 1 << 22;
constexpr int kAcceptLogitsMaxSeqs = 1 << 19;
size_t sd_spec_accept_workspace_size(int B, int k, int V, int mode) {
  if (B < 1 || B > kAcceptMaxSeqs || k < 1 || k > 16 || V < 1 || V > (1 << 18) ||
      (mode != SD_ACCEPT_GREEDY && mode != SD_ACCEPT_SAMPLED))
    return 0;
  return sd::accept_workspace_bytes(B, k, V, mode);
}

int sd_spec_accept(const float* p, const float* q, const int32_t* draft, const float* u,
                   int32_t* n_accepted, int32_t* tokens, int B, int k, int V, int mode,
                   void* workspace, size_t workspace_bytes, void* stream) {
  if (B < 1 || k < 1 || V < 1 || (mode != SD_ACCEPT_GREEDY && mode != SD_ACCEPT_SAMPLED))
    return SD_ERR_INVALID_ARG;
  if (k > 16 || V > (1 << 18) || B > kAcceptMaxSeqs) return SD_ERR_UNSUPPORTED;
  if (!p || !draft || !n_accepted || !tokens) return SD_ERR_INVALID_ARG;
  if (mode == SD_ACCEPT_SAMPLED && (!q || !u)) return SD_ERR_INVALID_ARG;
  if (!aligned(p, 4) || !aligned(draft, 4) || !aligned(n_accepted, 4) || !aligned(tokens, 4) ||
      (q && !aligned(q, 4)) || (u && !aligned(u, 4)))
    return SD_ERR_INVALID_ARG;
  const size_t need = sd::accept_workspace_bytes(B, k, V, mode);
  if (!workspace || workspace_bytes < need || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  sd::AcceptArgs a{};
  a.p = p;
  a.q = q;
  a.draft = draft;
  a.u = u;
  a.n_accepted = n_accepted;
  a.tokens = tokens;
  a.B = B;
  a.k = k;
  a.V = V;
  a.mode = mode;
  return status_from(sd::launch_accept(a, workspace, static_cast<hipStream_t>(stream)));
}

// ------------------------------------------- accept without allocation
int sd_spec_accept_noalloc(const float* p, const float* q, const int32_t* draft, const float* u,
                           int32_t* n_accepted, int32_t* tokens, int B, int k, int V, int mode, void* stream) {
  if (B < 1 || k < 1 || V < 1 || (mode != SD_ACCEPT_GREEDY && mode != SD_ACCEPT_SAMPLED))
    return SD_ERR_INVALID_ARG;
  if (k > 16 || V > (1 << 18)) return SD_ERR_UNSUPPORTED;
  if (!p || !draft || !n_accepted || !tokens) return SD_ERR_INVALID_ARG;
  if (mode == SD_ACCEPT_SAMPLED && (!q || !u)) return SD_ERR_INVALID_ARG;
  if (!aligned(p, 4) || !aligned(draft, 4) || !aligned(n_accepted, 4) || !aligned(tokens, 4) ||
      (q && !aligned(q, 4)) || (u && !aligned(u, 4)))
    return SD_ERR_INVALID_ARG;
  if (B > kScratchSeqs || sd::accept_partial_bytes(B, k, V, mode) > kScratchBytes - kScratchCounterBytes)
    return SD_ERR_WORKSPACE;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  unsigned char* base = nullptr;
  const hipError_t e = scratch_for_current_device(st, &base);
  if (e != hipSuccess) return status_from(e);
  sd::AcceptArgs a{};
  a.p = p;
  a.q = q;
  a.draft = draft;
  a.u = u;
  a.n_accepted = n_accepted;
  a.tokens = tokens;
  a.B = B;
  a.k = k;
  a.V = V;
  a.mode = mode;
  return status_from(sd::launch_accept_split(a, reinterpret_cast<unsigned*>(base), base + kScratchCounterBytes, st));
}

// ------------------------------------------------------ accept (logits)
size_t sd_spec_accept_logits_workspace_size(int B, int k, int V, int mode) {
  if (B < 1 || B > kAcceptLogitsMaxSeqs || k < 1 || k > 16 || V < 1 || V > (1 << 18) ||
      (mode != SD_ACCEPT_GREEDY && mode != SD_ACCEPT_SAMPLED))
    return 0;
  return sd::accept_logits_workspace_bytes(B, k, V, mode);
}

int sd_spec_accept_logits(const void* target_logits, const void* draft_logits, const int32_t* draft,
                          uint64_t seed, uint64_t offset, float temperature, int32_t* n_accepted,
                          int32_t* tokens, int B, int k, int V, int dtype, int mode, void* workspace,
                          size_t workspace_bytes, void* stream) {
  if (B < 1 || k < 1 || V < 1 || (mode != SD_ACCEPT_GREEDY && mode != SD_ACCEPT_SAMPLED) ||
      (dtype != SD_F32 && dtype != SD_BF16))
    return SD_ERR_INVALID_ARG;
  if (k > 16 || V > (1 << 18) || B > kAcceptLogitsMaxSeqs) return SD_ERR_UNSUPPORTED;
  if (!target_logits || !draft || !n_accepted || !tokens) return SD_ERR_INVALID_ARG;
  if (mode == SD_ACCEPT_SAMPLED && (!draft_logits || !isfinite(temperature) || !(temperature > 0.f)))
    return SD_ERR_INVALID_ARG;
  const size_t al = dtype == SD_F32 ? 4 : 2;
  if (!aligned(target_logits, al) || (draft_logits && !aligned(draft_logits, al)) || !aligned(draft, 4) ||
      !aligned(n_accepted, 4) || !aligned(tokens, 4))
    return SD_ERR_INVALID_ARG;
  const size_t need = sd::accept_logits_workspace_bytes(B, k, V, mode);
  if (!workspace || workspace_bytes < need || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  sd::AcceptLogitsArgs la{};
  la.rule.draft = draft;
  la.rule.n_accepted = n_accepted;
  la.rule.tokens = tokens;
  la.rule.B = B;
  la.rule.k = k;
  la.rule.V = V;
  la.rule.mode = mode;
  la.target_logits = target_logits;
  la.draft_logits = draft_logits;
  la.scale_log2 = mode == SD_ACCEPT_SAMPLED ? 1.4426950408889634f / temperature : 0.f;
  la.seed = seed;
  la.offset = offset;
  return status_from(sd::launch_accept_logits(la, dtype, workspace, static_cast<hipStream_t>(stream)));
}

int sd_philox_uniforms(uint64_t seed, uint64_t offset, float* u, int B, int n, void* stream) {
  if (!u || B < 1 || n < 1 || !aligned(u, 4)) return SD_ERR_INVALID_ARG;
  if (n > (1 << 16) || (long long)B * n > 2147483647LL) return SD_ERR_UNSUPPORTED;
  return status_from(sd::launch_philox_uniforms(seed, offset, u, B, n, static_cast<hipStream_t>(stream)));
}

// -------------------------------------------------------------- LM head
size_t sd_lm_head_workspace_size(int R, int d, int V, int dtype) {
  if (R < 1 || d < 1 || V < 1 || R > 4096 || V > (1 << 24) || (dtype != SD_F32 && dtype != SD_BF16))
    return 0;
  return sd::lm_head_workspace_bytes(R, V);
}

int sd_lm_head_probs(const void* hidden, const void* weight, float* probs, int R, int d, int V,
                     float temperature, int dtype, void* workspace, size_t workspace_bytes,
                     void* stream) {
  if (R < 1 || d < 1 || V < 1 || (dtype != SD_F32 && dtype != SD_BF16)) return SD_ERR_INVALID_ARG;
  if (!(temperature > 0.f) || !isfinite(temperature)) return SD_ERR_INVALID_ARG;
  if (!hidden || !weight || !probs || !aligned(probs, 4)) return SD_ERR_INVALID_ARG;
  if (R > 4096 || V > (1 << 24)) return SD_ERR_UNSUPPORTED;
  if (dtype == SD_BF16) {
    if (d % 64 != 0 || R > 256) return SD_ERR_UNSUPPORTED;
    if (!aligned(hidden, 16) || !aligned(weight, 16)) return SD_ERR_INVALID_ARG;
  } else if (!aligned(hidden, 4) || !aligned(weight, 4)) {
    return SD_ERR_INVALID_ARG;
  }
  const size_t need = sd::lm_head_workspace_bytes(R, V);
  if (!workspace || workspace_bytes < need || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  sd::LmHeadArgs a{};
  a.hidden = hidden;
  a.weight = weight;
  a.probs = probs;
  a.R = R;
  a.d = d;
  a.V = V;
  a.scale_log2 = 1.4426950408889634f / temperature;
  a.stats = static_cast<float*>(workspace);
  a.cus = device_cus();
  return status_from(sd::launch_lm_head(a, dtype, static_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------------- sampling
// T ~ Categorical(p) is the acceptance rule's final draw with no drafts:
// the acceptance kernels run with k = 0 (no tests; u[r] drives the draw).
size_t sd_sample_workspace_size(int R, int V) {
  if (R < 1 || V < 1 || V > (1 << 18)) return 0;
  const size_t acc = (sd::accept_workspace_bytes(R, 0, V, SD_ACCEPT_SAMPLED) + 15) / 16 * 16;
  return acc + (size_t)R * sizeof(int32_t);
}

int sd_sample_tokens(const float* probs, const float* u, int32_t* tokens, int R, int V,
                     void* workspace, size_t workspace_bytes, void* stream) {
  if (R < 1 || V < 1) return SD_ERR_INVALID_ARG;
  if (V > (1 << 18)) return SD_ERR_UNSUPPORTED;
  if (!probs || !u || !tokens || !aligned(probs, 4) || !aligned(u, 4) || !aligned(tokens, 4))
    return SD_ERR_INVALID_ARG;
  const size_t acc = (sd::accept_workspace_bytes(R, 0, V, SD_ACCEPT_SAMPLED) + 15) / 16 * 16;
  const size_t need = acc + (size_t)R * sizeof(int32_t);
  if (!workspace || workspace_bytes < need || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  sd::AcceptArgs a{};
  a.p = probs;
  a.q = nullptr;
  a.draft = nullptr;
  a.u = u;
  a.n_accepted = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + acc);
  a.tokens = tokens;
  a.B = R;
  a.k = 0;
  a.V = V;
  a.mode = SD_ACCEPT_SAMPLED;
  return status_from(sd::launch_accept(a, workspace, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

// ------------------------------------------------------------ draft layer
static bool linear_shape_ok(int R, int K, int N) {
  return R >= 1 && R <= 65535 && K >= 256 && K % 256 == 0 && K <= (1 << 20) && N >= 1 && N <= (1 << 24) &&
         (long long)R * N <= (1LL << 31);
}

size_t sd_linear_workspace_size(int R, int K, int N) {
  if (!linear_shape_ok(R, K, N)) return 0;
  return sd::plan_linear(R, K, N, device_cus()).part_bytes;
}

int sd_linear(const void* x, const void* w, const float* bias, const float* residual, float* y, int R, int K,
              int N, void* workspace, size_t workspace_bytes, void* stream) {
  if (R < 1 || K < 1 || N < 1 || !x || !w || !y) return SD_ERR_INVALID_ARG;
  if (!linear_shape_ok(R, K, N)) return SD_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y, 4) || (bias && !aligned(bias, 4)) ||
      (residual && !aligned(residual, 4)))
    return SD_ERR_INVALID_ARG;
  const sd::LinearPlan plan = sd::plan_linear(R, K, N, device_cus());
  if (!workspace || workspace_bytes < plan.part_bytes || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  sd::LinearArgs a{x, w, static_cast<float*>(workspace), R, K, N, plan.ksplit};
  hipError_t e = sd::launch_linear_partial(a, plan, st);
  if (e != hipSuccess) return status_from(e);
  return status_from(sd::launch_epi_add(a.part, plan.ksplit, R, N, bias, residual, y, st));
}

static bool semi_ar_shape_ok(int B, int r, int d, int Hq, int Hkv, int I, int Lmax, int* status) {
  *status = SD_ERR_INVALID_ARG;
  if (B < 1 || r < 1 || d < 1 || Hq < 1 || Hkv < 1 || I < 1 || Lmax < 1 || d % Hq != 0 || Hq % Hkv != 0)
    return false;
  *status = SD_ERR_UNSUPPORTED;
  const int D = d / Hq;
  if (r > 16 || (D != 64 && D != 128) || r * (Hq / Hkv) > 256 || d % 256 != 0 || I % 256 != 0 ||
      Lmax < r || (long long)B * r > 65535 || (long long)B * Lmax * Hkv * D > (1LL << 40))
    return false;
  *status = SD_OK;
  return true;
}

size_t sd_semi_ar_layer_workspace_size(int B, int r, int d, int num_q_heads, int num_kv_heads, int I,
                                       int Lmax) {
  int st;
  if (!semi_ar_shape_ok(B, r, d, num_q_heads, num_kv_heads, I, Lmax, &st)) return 0;
  const sd::SemiArPlan plan = sd::plan_semi_ar(B, r, d, num_q_heads, num_kv_heads, I, Lmax, device_cus());
  return plan.ok ? plan.workspace_bytes : 0;
}

int sd_semi_ar_layer(const void* u, const void* fc_w, const float* fc_b, const float* ln1, const void* wqkv,
                     const void* wo, const float* ln2, const void* wgu, const void* wdown, void* k_cache,
                     void* v_cache, const int32_t* pos, float* out, int B, int r, int d, int num_q_heads,
                     int num_kv_heads, int I, int Lmax, float eps, float theta, void* workspace,
                     size_t workspace_bytes, void* stream) {
  int st = SD_OK;
  if (!semi_ar_shape_ok(B, r, d, num_q_heads, num_kv_heads, I, Lmax, &st)) return st;
  if (!u || !fc_w || !fc_b || !ln1 || !wqkv || !wo || !ln2 || !wgu || !wdown || !k_cache || !v_cache || !pos ||
      !out || !isfinite(eps) || eps < 0.f || !isfinite(theta) || theta <= 0.f)
    return SD_ERR_INVALID_ARG;
  const void* a16[] = {u, fc_w, wqkv, wo, wgu, wdown, k_cache, v_cache};
  for (const void* p : a16)
    if (!aligned(p, 16)) return SD_ERR_INVALID_ARG;
  if (!aligned(fc_b, 4) || !aligned(ln1, 4) || !aligned(ln2, 4) || !aligned(pos, 4) || !aligned(out, 16))
    return SD_ERR_INVALID_ARG;
  const sd::SemiArPlan plan = sd::plan_semi_ar(B, r, d, num_q_heads, num_kv_heads, I, Lmax, device_cus());
  if (!plan.ok) return SD_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < plan.workspace_bytes || !aligned(workspace, 256)) return SD_ERR_WORKSPACE;
  sd::SemiArArgs a{};
  a.u = u;
  a.fc_w = fc_w;
  a.fc_b = fc_b;
  a.ln1 = ln1;
  a.wqkv = wqkv;
  a.wo = wo;
  a.ln2 = ln2;
  a.wgu = wgu;
  a.wdown = wdown;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.pos = pos;
  a.out = out;
  a.B = B;
  a.r = r;
  a.d = d;
  a.Hq = num_q_heads;
  a.Hkv = num_kv_heads;
  a.I = I;
  a.Lmax = Lmax;
  a.eps = eps;
  a.theta = theta;
  a.workspace = workspace;
  return status_from(sd::launch_semi_ar(a, plan, static_cast<hipStream_t>(stream)));
}

static bool semi_ar_draft_ok(int B, int r0, int d, int Hq, int Hkv, int I, int Lmax, int V, int K, int kp,
                             int* status) {
  if (!semi_ar_shape_ok(B, r0, d, Hq, Hkv, I, Lmax, status)) return false;
  *status = SD_ERR_INVALID_ARG;
  if (V < 1 || K < 1 || kp < 1 || kp > r0 || K % kp != 0) return false;
  *status = SD_ERR_UNSUPPORTED;
  if (kp > 8 || V > (1 << 18) || (long long)B * kp > 256 || (long long)B * K * V > (1LL << 40)) return false;
  if (K > kp && !semi_ar_shape_ok(B, 2 * kp, d, Hq, Hkv, I, Lmax, status)) return false;
  *status = SD_OK;
  return true;
}

size_t sd_semi_ar_draft_workspace_size(int B, int r0, int d, int num_q_heads, int num_kv_heads, int I, int Lmax,
                                       int V, int K, int k_prime) {
  int st;
  if (!semi_ar_draft_ok(B, r0, d, num_q_heads, num_kv_heads, I, Lmax, V, K, k_prime, &st)) return 0;
  const sd::SemiArDraftPlan plan =
      sd::plan_semi_ar_draft(B, r0, d, num_q_heads, num_kv_heads, I, Lmax, V, K, k_prime, device_cus());
  return plan.ok ? plan.workspace_bytes : 0;
}

int sd_semi_ar_draft(const void* u0, const void* fc_w, const float* fc_b, const float* ln1, const void* wqkv,
                     const void* wo, const float* ln2, const void* wgu, const void* wdown, const void* lm_w,
                     const void* emb, const void* ph, void* k_cache, void* v_cache, const int32_t* pos,
                     const float* u, int32_t* tokens, float* q, int B, int r0, int d, int num_q_heads,
                     int num_kv_heads, int I, int Lmax, int V, int K, int k_prime, float eps, float theta,
                     float temperature, void* workspace, size_t workspace_bytes, void* stream) {
  int st = SD_OK;
  if (!semi_ar_draft_ok(B, r0, d, num_q_heads, num_kv_heads, I, Lmax, V, K, k_prime, &st)) return st;
  if (!u0 || !fc_w || !fc_b || !ln1 || !wqkv || !wo || !ln2 || !wgu || !wdown || !lm_w || !emb || !ph ||
      !k_cache || !v_cache || !pos || !u || !tokens || !q || !isfinite(eps) || eps < 0.f || !isfinite(theta) ||
      theta <= 0.f || !isfinite(temperature) || !(temperature > 0.f))
    return SD_ERR_INVALID_ARG;
  const void* a16[] = {u0, fc_w, wqkv, wo, wgu, wdown, lm_w, emb, k_cache, v_cache};
  for (const void* p : a16)
    if (!aligned(p, 16)) return SD_ERR_INVALID_ARG;
  const void* a4[] = {fc_b, ln1, ln2, pos, u, tokens, q};
  for (const void* p : a4)
    if (!aligned(p, 4)) return SD_ERR_INVALID_ARG;
  if (!aligned(ph, 2)) return SD_ERR_INVALID_ARG;
  const sd::SemiArDraftPlan plan =
      sd::plan_semi_ar_draft(B, r0, d, num_q_heads, num_kv_heads, I, Lmax, V, K, k_prime, device_cus());
  if (!plan.ok) return SD_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < plan.workspace_bytes || !aligned(workspace, 256)) return SD_ERR_WORKSPACE;
  sd::SemiArDraftArgs a{};
  a.layer.u = u0;
  a.layer.fc_w = fc_w;
  a.layer.fc_b = fc_b;
  a.layer.ln1 = ln1;
  a.layer.wqkv = wqkv;
  a.layer.wo = wo;
  a.layer.ln2 = ln2;
  a.layer.wgu = wgu;
  a.layer.wdown = wdown;
  a.layer.k_cache = k_cache;
  a.layer.v_cache = v_cache;
  a.layer.pos = pos;
  a.layer.B = B;
  a.layer.r = r0;
  a.layer.d = d;
  a.layer.Hq = num_q_heads;
  a.layer.Hkv = num_kv_heads;
  a.layer.I = I;
  a.layer.Lmax = Lmax;
  a.layer.eps = eps;
  a.layer.theta = theta;
  a.lm_w = lm_w;
  a.emb = emb;
  a.ph = ph;
  a.u = u;
  a.tokens = tokens;
  a.q = q;
  a.V = V;
  a.K = K;
  a.kp = k_prime;
  a.temperature = temperature;
  a.workspace = workspace;
  return status_from(sd::launch_semi_ar_draft(a, plan, static_cast<hipStream_t>(stream)));
}

int sd_linear_q8(const void* x, const int8_t* wq, const float* scale, const float* bias, const float* residual,
                 float* y, int R, int K, int N, void* workspace, size_t workspace_bytes, void* stream) {
  if (!scale || !aligned(scale, 4)) return SD_ERR_INVALID_ARG;
  if (R < 1 || K < 1 || N < 1 || !x || !wq || !y) return SD_ERR_INVALID_ARG;
  if (!linear_shape_ok(R, K, N)) return SD_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(wq, 16) || !aligned(y, 4) || (bias && !aligned(bias, 4)) ||
      (residual && !aligned(residual, 4)))
    return SD_ERR_INVALID_ARG;
  const sd::LinearPlan plan = sd::plan_linear(R, K, N, device_cus());
  if (!workspace || workspace_bytes < plan.part_bytes || !aligned(workspace, 16)) return SD_ERR_WORKSPACE;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  sd::LinearArgs a{x, wq, static_cast<float*>(workspace), R, K, N, plan.ksplit, scale};
  hipError_t e = sd::launch_linear_partial(a, plan, st);
  if (e != hipSuccess) return status_from(e);
  return status_from(sd::launch_epi_add(a.part, plan.ksplit, R, N, bias, residual, y, st));
}

int sd_semi_ar_layer_q8(const void* u, const int8_t* fc_w, const float* fc_s, const float* fc_b, const float* ln1,
                        const int8_t* wqkv, const float* wqkv_s, const int8_t* wo, const float* wo_s,
                        const float* ln2, const int8_t* wgu, const float* wgu_s, const int8_t* wdown,
                        const float* wdown_s, void* k_cache, void* v_cache, const int32_t* pos, float* out, int B,
                        int r, int d, int num_q_heads, int num_kv_heads, int I, int Lmax, float eps, float theta,
                        void* workspace, size_t workspace_bytes, void* stream) {
  const float* sc[] = {fc_s, wqkv_s, wo_s, wgu_s, wdown_s};
  int st = SD_OK;
  if (!semi_ar_shape_ok(B, r, d, num_q_heads, num_kv_heads, I, Lmax, &st)) return st;
  for (const float* p : sc)
    if (!p || !aligned(p, 4)) return SD_ERR_INVALID_ARG;
  if (!u || !fc_w || !fc_b || !ln1 || !wqkv || !wo || !ln2 || !wgu || !wdown || !k_cache || !v_cache || !pos ||
      !out || !isfinite(eps) || eps < 0.f || !isfinite(theta) || theta <= 0.f)
    return SD_ERR_INVALID_ARG;
  const void* a16[] = {u, fc_w, wqkv, wo, wgu, wdown, k_cache, v_cache};
  for (const void* p : a16)
    if (!aligned(p, 16)) return SD_ERR_INVALID_ARG;
  if (!aligned(fc_b, 4) || !aligned(ln1, 4) || !aligned(ln2, 4) || !aligned(pos, 4) || !aligned(out, 16))
    return SD_ERR_INVALID_ARG;
  const sd::SemiArPlan plan = sd::plan_semi_ar(B, r, d, num_q_heads, num_kv_heads, I, Lmax, device_cus());
  if (!plan.ok) return SD_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < plan.workspace_bytes || !aligned(workspace, 256)) return SD_ERR_WORKSPACE;
  sd::SemiArArgs a{};
  a.u = u;
  a.fc_w = fc_w;
  a.fc_b = fc_b;
  a.ln1 = ln1;
  a.wqkv = wqkv;
  a.wo = wo;
  a.ln2 = ln2;
  a.wgu = wgu;
  a.wdown = wdown;
  a.fc_s = fc_s;
  a.wqkv_s = wqkv_s;
  a.wo_s = wo_s;
  a.wgu_s = wgu_s;
  a.wdown_s = wdown_s;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.pos = pos;
  a.out = out;
  a.B = B;
  a.r = r;
  a.d = d;
  a.Hq = num_q_heads;
  a.Hkv = num_kv_heads;
  a.I = I;
  a.Lmax = Lmax;
  a.eps = eps;
  a.theta = theta;
  a.workspace = workspace;
  return status_from(sd::launch_semi_ar(a, plan, static_cast<hipStream_t>(stream)));
}

int sd_avg_pool_compress(const void* feats, float* out, int B, int N, int C, int d, int dtype, void* stream) {
  if (B < 1 || N < 1 || C < 1 || d < 1 || C > N || (dtype != SD_F32 && dtype != SD_BF16)) return SD_ERR_INVALID_ARG;
  if (!feats || !out || !aligned(feats, dtype == SD_F32 ? 4 : 2) || !aligned(out, 4)) return SD_ERR_INVALID_ARG;
  if (B > 65535 || C > 65535 || N > (1 << 24) || d > (1 << 20)) return SD_ERR_UNSUPPORTED;
  return status_from(sd::launch_avg_pool(feats, out, B, N, C, d, dtype, static_cast<hipStream_t>(stream)));
}
