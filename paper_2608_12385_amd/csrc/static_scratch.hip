// The grouped decode step without any device memory of the caller's beyond
// its inputs, outputs, weights and cache: the step's buffers (activations,
// split partials, logits and their statistics, MoE lists) live in one static
// device array of the library, `scratch`, instead of the model workspace's
// step region.  Meant for callers that cannot allocate while they step.
//
// Each GPU holds its own copy of the array from the library's load until the
// process ends; its address on a device is taken once, with that device
// current, by hipGetSymbolAddress and kept per device.  Host code uses only
// that address, never the array's name.  Every call on one GPU shares that
// GPU's array: calls that overlap on one GPU (other streams, other threads,
// other models) race.  Nothing in it needs clearing between calls: every
// element a step reads is written earlier in the same step, except padding
// rows whose results are never used.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/dbt.h"
#include "host_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;  // DBT_STATIC_SCRATCH_BYTES
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch`, per device

// Address of the array on the current device (taken on first use).
dbt_status scratch_address(void **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return dbt::set_error(DBT_ERR_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return dbt::set_error(DBT_ERR_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return dbt::set_error(DBT_ERR_HIP, hipGetErrorString(e));
    if (!p) return dbt::set_error(DBT_ERR_HIP, "no device address for the static scratch");
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return DBT_OK;
}

}  // namespace

static_assert(kScratchBytes == DBT_STATIC_SCRATCH_BYTES, "public size and array size differ");

extern "C" dbt_status dbt_decode_step_noalloc(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on,
                                              dbt_step_out *out, dbt_stream stream) {
  if (!m) return dbt::set_error(DBT_ERR_ARG, "model is NULL");
  const size_t need = dbt::step_bytes(m);
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof msg, "the model's step buffers need %zu bytes; the static scratch holds %zu", need,
             kScratchBytes);
    return dbt::set_error(DBT_ERR_UNSUPPORTED, msg);
  }
  void *ptr = nullptr;
  const dbt_status s = scratch_address(&ptr);
  if (s) return s;
  return dbt::decode_step_in(m, kv, in, branch_on, out, stream, (char *)ptr);
}
