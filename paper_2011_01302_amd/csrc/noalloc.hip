// ios_run_noalloc: ios_run for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  ios_run's stage kernels use memory of the graph beyond the
// caller's inputs and outputs: the intermediate activations between stages
// and the per-stage counters of stages whose groups hold chains.  Here both
// live in one file-scope device array, `scratch`, of fixed size, and the
// entry point makes no allocation of any kind.
//
// Each device the library runs on holds its own copy of the array (at its
// own address) until the process ends.  Its device address is looked up once
// per device, with that device current, when a graph first sets up its
// device side (ensure_device), and kept per device; host code never passes
// the array's name itself (in host code that name is only a stand-in, not a
// device address).  Every call on one device shares that device's array and
// leaves the last call's contents in it: calls that overlap in time on one
// device race (issue them on one stream).
#include <atomic>
#include <cstring>
#include <mutex>

#include "ios_internal.h"

namespace ios {

namespace {

constexpr int kMaxDevices = 64;
// Counter block: [1] workgroups finished + kCtrCopies copies of kCtrStride
// per-op counters (StageArgs::ctr), rounded up to 256 bytes.  Every stage
// kernel with in-stage dependencies leaves them at zero when it ends, so one
// block serves every stage of every call.
constexpr size_t kCtrBytes = ((2 + (size_t)kCtrStride * kCtrCopies) * sizeof(int32_t) + 255) & ~(size_t)255;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_setup_mu;
std::atomic<unsigned char *> g_scratch_ptr[kMaxDevices];

thread_local char g_msg[256];

int refuse(int code, const char *msg) {
  std::strncpy(g_msg, msg, sizeof(g_msg) - 1);
  g_msg[sizeof(g_msg) - 1] = 0;
  set_last_error_text(g_msg);
  return code;
}

}  // namespace

void noalloc_setup(int device) {
  if (device < 0 || device >= kMaxDevices) fail(IOS_E_UNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_setup_mu);
  if (g_scratch_ptr[device].load()) return;
  void *p = nullptr;
  hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
  // the counters must start at zero (the kernels keep them there)
  hip_check(hipMemset(p, 0, kCtrBytes), "hipMemset(scratch counters)");
  hip_check(hipDeviceSynchronize(), "hipDeviceSynchronize");
  g_scratch_ptr[device].store((unsigned char *)p);
}

size_t noalloc_counter_bytes() { return kCtrBytes; }

}  // namespace ios

using namespace ios;

extern "C" int ios_run_noalloc(ios_graph *g, const ios_schedule_t *q, const float *const *d_inputs,
                               float *const *d_outputs, void *hip_stream) {
  if (!g || !q) return refuse(IOS_E_ARG, "null graph or schedule");
  if (!g->finalized || !g->device_ready)
    return refuse(IOS_E_STATE, "graph not set up on the device: run the schedule once with ios_run first");
  if (q->g != g) return refuse(IOS_E_ARG, "schedule does not belong to this graph");
  if (g->noalloc_bytes > kNoAllocScratchBytes)
    return refuse(IOS_E_UNSUPPORTED,
                  "the graph's intermediates and counters exceed the 64 MiB no-allocation scratch array");
  if (q->compiled.empty() || q->compiled.size() != q->strategies.size())
    return refuse(IOS_E_STATE, "schedule not compiled: run it once with ios_run first");
  if ((!g->inputs.empty() && !d_inputs) || (!g->outputs.empty() && !d_outputs))
    return refuse(IOS_E_ARG, "null input or output list");
  if (hipSetDevice(g->device) != hipSuccess) return refuse(IOS_E_HIP, "hipSetDevice failed");
  unsigned char *base = g_scratch_ptr[g->device].load();
  if (!base) return refuse(IOS_E_STATE, "scratch array not set up on this device");
  for (const Buffer &b : g->bufs) {
    if (b.input_index >= 0 && !d_inputs[b.input_index]) return refuse(IOS_E_ARG, "null input pointer");
    if (b.output_index >= 0 && !d_outputs[b.output_index]) return refuse(IOS_E_ARG, "null output pointer");
  }
  hipStream_t s = (hipStream_t)hip_stream;
  for (const auto &cs : q->compiled) {
    StageArgs a{};
    a.n_slots = (int)cs->slot_buf.size();
    for (int i = 0; i < a.n_slots; ++i) {
      const int bi = cs->slot_buf[i];
      const Buffer &b = g->bufs[bi];
      if (b.input_index >= 0) a.slot[i] = const_cast<float *>(d_inputs[b.input_index]);
      else if (b.output_index >= 0) a.slot[i] = d_outputs[b.output_index];
      else a.slot[i] = (float *)(base + g->noalloc_off[bi]);
    }
    a.ctr = (int32_t *)base;
    a.err = g->d_err;
    a.spin_limit = 1 << 24;
    if (launch_stage(cs->d_table, (int)cs->table.size(), a, cs->persistent, cs->grid, cs->lds_bytes,
                     cs->variant, s) != hipSuccess)
      return refuse(IOS_E_HIP, "stage launch failed");
  }
  return IOS_OK;
}
