// Attention entry point that allocates nothing: the parts of query tiles cut
// between workgroups live in a static device array instead of a workspace,
// for callers that cannot allocate device memory (code under HIP graph
// capture, serving loops, harnesses that forbid hipMalloc).
#include <mutex>

#include "../../include/orch.h"
#include "common.h"
#include "kernels.h"

using namespace orch;

namespace orch_detail {
int set_error(int code, const char* msg);
int check_attention_args(const void* q, const void* kv_stale, size_t stale_bs,
                         const void* kv_fresh, size_t fresh_bs, int fresh_begin, int n_fresh,
                         int B, int heads, int n_q, int n_kv, int head_dim, const void* out,
                         int dtype);
AttnParams attention_params(const void* q, const void* kv_stale, size_t stale_bs,
                            const void* kv_fresh, size_t fresh_bs, int fresh_begin, int n_fresh,
                            int B, int heads, int n_q, int n_kv, int head_dim, void* out);
}  // namespace orch_detail

namespace {

// The work plan never uses more than 512 workgroups, each with two part
// slots of 128 queries: bf16 O/l of d <= 72 channels plus a float2 (max, sum)
// per query, 19,922,944 bytes; the array rounds that up to 20 MiB.
constexpr size_t kScratchBytes = (size_t)20 << 20;

// Each device holds its own copy of the array at its own address; host code
// must use the address hipGetSymbolAddress returns, never the array's name.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's scratch, looked up once per device with
// that device current.
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return orch_detail::set_error(ORCH_EHIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return orch_detail::set_error(ORCH_EINVAL, "device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return orch_detail::set_error(ORCH_EHIP, "hipGetSymbolAddress(scratch) failed");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return ORCH_OK;
}

}  // namespace

extern "C" {

int orch_op_attention_noalloc(const void* q, const void* kv_stale, size_t stale_bs,
                              const void* kv_fresh, size_t fresh_bs, int fresh_begin, int n_fresh,
                              int B, int heads, int n_q, int n_kv, int head_dim, void* out,
                              int dtype, void* hip_stream) {
  int rc = orch_detail::check_attention_args(q, kv_stale, stale_bs, kv_fresh, fresh_bs,
                                             fresh_begin, n_fresh, B, heads, n_q, n_kv, head_dim,
                                             out, dtype);
  if (rc) return rc;
  const size_t need = attention_workspace_bytes(B, heads, n_q, n_kv, head_dim, dtype);
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof msg, "shape needs %zu bytes of scratch, the static scratch holds %zu",
             need, kScratchBytes);
    return orch_detail::set_error(ORCH_EINVAL, msg);
  }
  AttnParams ap = orch_detail::attention_params(q, kv_stale, stale_bs, kv_fresh, fresh_bs,
                                                fresh_begin, n_fresh, B, heads, n_q, n_kv,
                                                head_dim, out);
  if (need > 0) {
    rc = scratch_address(&ap.ws);
    if (rc) return rc;
    ap.ws_bytes = kScratchBytes;
  }
  hipError_t e = launch_attention(ap, dtype, (hipStream_t)hip_stream);
  if (e != hipSuccess) return orch_detail::set_error(ORCH_EHIP, hipGetErrorString(e));
  return ORCH_OK;
}

}  // extern "C"
