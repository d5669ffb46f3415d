// ss_simulate_batch_noalloc: the simulation of ss_simulate_batch for callers
// that cannot allocate device memory (code under HIP graph capture, tight
// serving loops, harnesses that forbid allocation).  Its scratch is one
// file-scope device array per GPU, kNoAllocScratch bytes, held from the first
// use on that GPU until the process ends; every call on a GPU shares it.
#include <mutex>

#include "ss_internal.h"

namespace {

constexpr size_t kNoAllocScratch = size_t(128) << 20;
constexpr int kMaxDev = 256;

// In host code the name `scratch` stands for the symbol, not a device
// address: the per-device address comes from hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratch];

std::mutex g_mu;
void *g_addr[kMaxDev];  // address of `scratch` on each device, once taken

// The device address of `scratch` on the current device (taken once).
int scratch_address(int device, void **out) {
  if (device < 0 || device >= kMaxDev) return ss_set_error(SS_ERR_UNSUPPORTED, "device id beyond 255");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return ss_set_error(SS_ERR_DEVICE, std::string("hipGetSymbolAddress of the fixed scratch: ") +
                                             hipGetErrorString(e));
    g_addr[device] = p;
  }
  *out = g_addr[device];
  return SS_OK;
}

}  // namespace

extern "C" int ss_simulate_batch_noalloc(const ss_gmg *g, const uint8_t *placements, int64_t B, int layout,
                                         int64_t *out_makespan, int64_t *out_peak_mem, uint8_t *out_violation,
                                         int64_t *out_sla_slack, int64_t *out_sumfin, void *hip_stream) {
  ss_clear_error();
  if (!g) return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_noalloc: g is NULL");
  int64_t need = 0;
  // the same checks as ss_simulate_batch, and the smallest scratch this call needs
  int rc = ss_simulate_workspace_size(g, B, layout, &need, nullptr);
  if (rc != SS_OK) return rc;
  if (B == 0) return SS_OK;
  if (!out_makespan || !out_violation)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_noalloc: out_makespan and out_violation are required");
  if (!placements && g->n_ops > 0)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_noalloc: placements is NULL");
  if ((size_t)need > kNoAllocScratch)
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_simulate_batch_noalloc: this batch needs at least " +
                                                std::to_string(need) + " bytes of scratch, more than the fixed " +
                                                std::to_string(kNoAllocScratch));
  void *ws = nullptr;
  rc = scratch_address(g->device, &ws);
  if (rc != SS_OK) return rc;
  SsPlace src;
  src.p = placements;
  src.B = B;
  src.op_major = (layout & SS_LAYOUT_OP_MAJOR) != 0;
  SsWork W;
  W.ptr = ws;
  W.bytes = kNoAllocScratch;
  W.single = true;
  return ss_run_simulate(g, src, out_makespan, out_peak_mem, out_violation, out_sla_slack, out_sumfin,
                         static_cast<hipStream_t>(hip_stream), (layout & SS_DISPATCH_READY) != 0,
                         (layout & SS_LINK_PORTS) != 0, W);
}
