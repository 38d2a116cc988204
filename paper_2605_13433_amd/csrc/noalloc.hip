// The attention forward for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// allocation): the same kernels as hstu_jagged_attn_fwd, with the workspace
// replaced by one fixed device array per GPU.
//
// The forward's workspace holds the control words (list length, pop
// counter, contract status), the per-sequence records and the work list;
// the scheduler kernel of every call rewrites each word the later kernels
// read, so nothing has to be cleared between calls.  Calls on one GPU share
// its array: two calls that overlap on that GPU (on different streams, or
// from different threads) race on it.
#include <mutex>

#include "internal.h"

namespace hstu {

namespace {

constexpr size_t SCRATCH_BYTES = HSTU_NOALLOC_SCRATCH_BYTES;
constexpr int MAX_DEVICES = 64;

// Device-side storage.  In host code `scratch` names a host-side stand-in,
// not the device array: host code passes only the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

std::mutex g_mu;
void *g_addr[MAX_DEVICES];      // the array's address on each device, once looked up

// Address of the array on device `dev` (the current device), looked up on
// the first call on that device.  No allocation: the array is part of the
// library's code object, loaded with it onto every device it runs on.
void *scratch_addr(int dev) {
  if (dev < 0 || dev >= MAX_DEVICES) {
    fail(HSTU_ENOTSUP, "device %d: the no-allocation entry point supports devices 0..%d",
         dev, MAX_DEVICES - 1);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
      return nullptr;
    }
    g_addr[dev] = p;
  }
  return g_addr[dev];
}

}  // namespace

}  // namespace hstu

extern "C" int hstu_jagged_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                                            const void *u, const int64_t *seq_offsets,
                                            int32_t B, int32_t max_len, int32_t H, int32_t d,
                                            const hstu_rab *rab, hstu_fwd_out *out,
                                            void *stream) {
  static const hstu::FixedScratch fixed{hstu::scratch_addr, hstu::SCRATCH_BYTES};
  return hstu::attn_fwd_call(q, k, v, u, seq_offsets, B, max_len, H, d, rab, out, stream,
                             &fixed);
}
