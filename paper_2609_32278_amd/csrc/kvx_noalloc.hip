// extend_attention_noalloc: extend_attention for callers that cannot allocate
// device memory during the call (tight serving loops, harnesses that forbid
// hipMalloc).  It is not capturable into a HIP graph: the plan is built on the
// host per call and copied from a host vector freed when the call returns.
//
// The work plan and the partial results of split key ranges go into one fixed
// device array, `scratch`, instead of the pool's staging buffer and growable
// workspace; the kernels are the same ones extend_attention launches.  Every GPU
// the library runs on holds its own copy of the array until the process ends.
// In host code the array's name is only a host-side stand-in: its device address
// on each GPU is looked up once with hipGetSymbolAddress (that GPU current) and
// only that address is ever passed to a copy or a kernel.

#include <mutex>

#include "kvx_internal.h"

namespace {

constexpr size_t kPlanBytes = KVX_NOALLOC_PLAN_BYTES;
constexpr size_t kPartsBytes = KVX_NOALLOC_PARTS_BYTES;
static_assert(kPlanBytes % 256 == 0, "the partial-result region starts 256-byte aligned");

__device__ __align__(256) uint8_t scratch[kPlanBytes + kPartsBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_base[kMaxDevices] = {};

// Device address of `scratch` on `device`, which the caller has made current.
int scratch_address(int device, void** base) {
  if (device < 0 || device >= kMaxDevices)
    return kvx::report(KVX_EUNSUPPORTED, "device %d: the allocation-free entry point covers devices 0..%d", device,
                       kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_base[device] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return kvx::report(KVX_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", device, hipGetErrorString(e));
    g_base[device] = p;
  }
  *base = g_base[device];
  return KVX_OK;
}

const kvx::FixedScratch kScratch{kPlanBytes, kPartsBytes, scratch_address};

}  // namespace

extern "C" int extend_attention_noalloc(kvx_pool* pool, const kvx_batch* batch, const void* q, int32_t num_q_heads,
                                        float sm_scale, void* out, float* lse, kvx_stream_t stream) {
  return kvx::attention_call(pool, batch, q, num_q_heads, sm_scale, out, lse, stream, &kScratch);
}
