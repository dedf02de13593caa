// zl_kernel_attention_bwd_noalloc: the attention backward of
// zl_kernel_attention (backward = 1) for callers that cannot allocate device
// memory.  Its one scratch buffer -- delta[b, h, i] = sum_d dO . O, the row
// term of the softmax backward, B * Hq * S floats -- lives in a file-scope
// device array instead of a caller buffer, so the call allocates nothing.
//
// The array is a symbol of this library's code object: each GPU the library
// runs on holds its own copy at its own address until the process ends.
// Host code never passes the symbol itself to a kernel (its host-side name
// is not a device address); the address is looked up once per device with
// hipGetSymbolAddress and kept.  Every call on one GPU shares that GPU's
// array: calls that overlap on one GPU (on different streams, or from
// different threads without ordering) race on it.  The delta kernel writes
// every entry it later reads, so nothing has to start at zero.
#include <math.h>
#include <string.h>

#include <mutex>
#include <string>

#include "../../include/zl_inspect.h"
#include "internal.h"
#include "common.h"

namespace {

constexpr size_t NOALLOC_DELTA_MAX = (size_t)1 << 20;  // floats (4 MiB): B * Hq * S
constexpr int MAX_DEVICES = 64;

__device__ __align__(256) float scratch[NOALLOC_DELTA_MAX];

std::mutex g_mu;
float* g_scratch[MAX_DEVICES];  // device address of `scratch`, per device

// The current device's address of `scratch`, looked up on its first use.
hipError_t scratch_ptr(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = static_cast<float*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" zl_status zl_kernel_attention_bwd_noalloc(int B, int S, int Hq, int Hkv, int hd,
                                                     const void* q, const void* k, const void* v,
                                                     int64_t ld_qkv, const int32_t* seq_lens,
                                                     const void* o, const float* lse,
                                                     const void* dout, void* dq, void* dk, void* dv,
                                                     int dtype, void* stream) {
  using namespace zl;
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || !q || !k || !v || !o || !lse ||
      !seq_lens || !dout || !dq || !dk || !dv)
    return set_error(ZL_ERR_INVALID_ARG, "bad attention args");
  if (hd != 16 && hd != 32 && hd != 64 && hd != 128)
    return set_error(ZL_ERR_UNSUPPORTED, "head_dim must be 16, 32, 64 or 128");
  if (dtype != ZL_F32 && dtype != ZL_BF16) return set_error(ZL_ERR_INVALID_ARG, "bad dtype");
  if ((size_t)B * Hq * S > NOALLOC_DELTA_MAX)
    return set_error(ZL_ERR_UNSUPPORTED,
                     "B * Hq * S = " + std::to_string((size_t)B * Hq * S) +
                         " exceeds the no-allocation scratch of " +
                         std::to_string(NOALLOC_DELTA_MAX) + " floats");
  float* delta = nullptr;
  hipError_t e = scratch_ptr(&delta);
  if (e != hipSuccess)
    return set_error(ZL_ERR_HIP, std::string("scratch address: ") + hipGetErrorString(e));
  AttnDesc a;
  memset(&a, 0, sizeof(a));
  a.B = B; a.S = S; a.Hq = Hq; a.Hkv = Hkv; a.hd = hd;
  a.q = q; a.k = k; a.v = v; a.ldq = a.ldk = a.ldv = ld_qkv;
  a.o = const_cast<void*>(o); a.ldo = (int64_t)Hq * hd; a.lse = const_cast<float*>(lse);
  a.seq_lens = seq_lens;
  a.dout = dout; a.lddo = (int64_t)Hq * hd; a.delta = delta;
  a.dq = dq; a.dk = dk; a.dv = dv; a.lddq = a.lddk = a.lddv = ld_qkv;
  a.scale = 1.f / sqrtf((float)hd);
  bool fused = false;
  e = launch_attn_bwd(a, dtype == ZL_BF16 ? BF16 : F32, reinterpret_cast<hipStream_t>(stream),
                      &fused);
  if (e != hipSuccess) return set_error(ZL_ERR_HIP, std::string("attention backward: ") +
                                                        hipGetErrorString(e));
  return ZL_OK;
}
