// osprey_verify_rows_static: the stateless verification of osprey_verify_rows for
// callers that cannot allocate device memory and hold no drafter handle.  Every
// scratch buffer of the verification kernels -- the inverse vocabulary map, the chunk
// records, the residual sums, the per-sequence state and the device error word --
// lives in one file-scope device array of fixed size instead of a workspace.
//
// Each GPU holds its own copy of `scratch` (loaded with the code object) until the
// process ends.  Host code never uses the array's name as an address: the first call
// on a device looks its device address up (hipGetSymbolAddress, with that device
// current) and keeps it per device.  Calls on one GPU share the array, so calls that
// overlap on one GPU (two streams, two host threads) race; each call clears what must
// start at zero (the error word) and rebuilds the inverse map.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "../../include/osprey.h"
#include "internal.h"

#define OSPREY_API extern "C" __attribute__((visibility("default")))

namespace osp {
namespace {

// Limits of one call (the scratch array is sized for them: about 7.4 MB).
constexpr int kStaticMaxBatch = 64;
constexpr int kStaticMaxK = 16;
constexpr int kStaticMaxVocab = 262144;
constexpr int kSChunk = 4096;                      // ids per verification chunk
constexpr long align256(long x) { return (x + 255) & ~255L; }
// layout of the scratch array for the largest call it serves
constexpr long kOffT2d = 0;
constexpr long kOffPart = align256(kOffT2d + 4L * kStaticMaxVocab);
constexpr long kMaxChunks = (kStaticMaxVocab + kSChunk - 1) / kSChunk;
constexpr long kOffRes = align256(kOffPart + 16L * kStaticMaxBatch * (2L * kStaticMaxK + 1) * kMaxChunks);
constexpr long kOffSub = align256(kOffRes + 16L * kStaticMaxBatch * kMaxChunks);
constexpr long kOffState = align256(kOffSub + 16L * kVSub * kStaticMaxBatch * kMaxChunks);
constexpr long kOffStat = align256(kOffState + 16L * kStaticMaxBatch);
constexpr long kOffErr = align256(kOffStat + 32L * kStaticMaxBatch);
constexpr long kScratchBytes = align256(kOffErr + 16);

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` per device, looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// The message goes to osprey_last_error() like every other call's.
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return report_error(code, buf);
}

// Prepares the call: the inverse map t2d = -1 everywhere, then t2d[d2t[i]] = i for the
// mapped rows (the largest row on a collision: deterministic, and for the injective
// maps the contract requires, the one row), and a zero error word.
__global__ void k_static_clear(int32_t* t2d, int V_T, uint32_t* err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < V_T) t2d[i] = -1;
  if (i == 0) err[0] = 0u;
}

__global__ void k_static_invert(const int32_t* d2t, int V_d, int32_t* t2d, int V_T) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= V_d) return;
  const int t = d2t[i];
  if (t >= 0 && t < V_T) atomicMax(t2d + t, i);   // entries outside [0, V_T) stay unmapped
}

}  // namespace
}  // namespace osp

using namespace osp;

OSPREY_API int osprey_verify_rows_static(const osprey_verify_rows_args* a, const int32_t* d2t,
                                         int32_t vocab_draft, int32_t vocab_target, void* hip_stream) {
  if (!a || !d2t) return fail(OSPREY_E_INVALID, "args and d2t must be non-NULL");
  const int B = a->batch, K = a->K;
  if (B < 1 || B > kStaticMaxBatch) return fail(OSPREY_E_CAPACITY, "batch %d not in [1, %d]", B, kStaticMaxBatch);
  if (K < 0 || K > kStaticMaxK) return fail(OSPREY_E_CAPACITY, "K %d not in [0, %d]", K, kStaticMaxK);
  if (vocab_draft < 1 || vocab_draft > kStaticMaxVocab || vocab_target < 1 || vocab_target > kStaticMaxVocab)
    return fail(OSPREY_E_CAPACITY, "vocabularies %d / %d not in [1, %d]", vocab_draft, vocab_target,
                kStaticMaxVocab);
  if (!a->target_logits || !a->temperature || !a->u_bonus || !a->accept_len || !a->accept_mask ||
      !a->out_tokens || (K > 0 && (!a->draft_logits || !a->draft_tokens || !a->u_accept)))
    return fail(OSPREY_E_INVALID, "a verify pointer is NULL");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(OSPREY_E_DEVICE, "no current HIP device (or device index beyond %d)", kMaxDevices);
  char* base;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
      void* p = nullptr;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(OSPREY_E_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      g_ptr[dev] = p;
    }
    base = static_cast<char*>(g_ptr[dev]);
  }
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  VerifyArgs v{};
  v.B = B;
  v.K = K;
  v.target = a->target_logits;
  v.draft = a->draft_logits;
  v.ld_draft_b = K;
  v.drafts = a->draft_tokens;
  v.ld_drafts = K;
  v.temp = a->temperature;
  v.temp_d = a->draft_temperature ? a->draft_temperature : a->temperature;
  v.u_acc = a->u_accept;
  v.u_bonus = a->u_bonus;
  v.d2t = d2t;
  v.t2d = reinterpret_cast<int32_t*>(base + kOffT2d);
  v.V_T = vocab_target;
  v.V_d = vocab_draft;
  v.chunk = kSChunk;
  v.nchunk_t = (vocab_target + kSChunk - 1) / kSChunk;
  v.nchunk_d = (vocab_draft + kSChunk - 1) / kSChunk;
  v.part = reinterpret_cast<float*>(base + kOffPart);
  v.res_part = reinterpret_cast<double*>(base + kOffRes);
  v.res_sub = reinterpret_cast<double*>(base + kOffSub);
  v.vstate = reinterpret_cast<int32_t*>(base + kOffState);
  v.vstat = reinterpret_cast<double*>(base + kOffStat);
  v.err = reinterpret_cast<uint32_t*>(base + kOffErr);
  v.accept_len = a->accept_len;
  v.accept_mask = a->accept_mask;
  v.out_tokens = a->out_tokens;
  hipLaunchKernelGGL(k_static_clear, dim3((vocab_target + 255) / 256), dim3(256), 0, st,
                     const_cast<int32_t*>(v.t2d), vocab_target, v.err);
  hipLaunchKernelGGL(k_static_invert, dim3((vocab_draft + 255) / 256), dim3(256), 0, st, d2t, vocab_draft,
                     const_cast<int32_t*>(v.t2d), vocab_target);
  launch_verify(v, st);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(OSPREY_E_DEVICE, "kernel launch: %s", hipGetErrorString(e));
  return report_error(OSPREY_OK, "");
}
