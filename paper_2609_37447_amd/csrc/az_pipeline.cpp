// Host submission pipeline in front of az_eval_batch.
//
// The paper finds that batching alone does not keep its GPUs busy: host-side
// preparation and submission must overlap GPU execution, through preallocated
// staging buffers, asynchronous copies, completion events and graph replay
// (Section 5.2 "Batching and host-side submission").  A pipeline owns `slots`
// independent slots on one device; each slot has pinned host buffers (written
// and read by the caller), device buffers, its own stream and a completion
// event.  Submitting a slot enqueues copy-in, evaluation and copy-out on the
// slot's stream and returns at once, so the copies of one slot overlap the
// evaluation of another.  With graphs enabled the three steps of a slot are
// captured once per batch size and replayed.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <new>
#include <vector>

#include "az.h"
#include "az_internal.h"

struct az_pipeline {
  struct Slot {
    float* h_planes = nullptr;
    uint8_t* h_legal = nullptr;
    float* h_policy = nullptr;
    float* h_value = nullptr;
    float* d_planes = nullptr;
    uint8_t* d_legal = nullptr;
    float* d_policy = nullptr;
    float* d_value = nullptr;
    hipStream_t stream = nullptr;
    hipEvent_t done = nullptr;
    hipGraphExec_t exec = nullptr;
    int graph_b = 0;
    bool submitted = false;
  };
  az_net* net = nullptr;
  int device = 0;
  int max_batch = 0, in_planes = 0, n_moves = 0;
  bool graphs = false;
  std::vector<Slot> slots;
};

namespace {

int hip_err(hipError_t e, const char* what) {
  (void)hipGetLastError();
  return az_fail(e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation ? AZ_ERR_NOMEM : AZ_ERR_DEVICE, what);
}

void release(az_pipeline* p) {
  for (auto& s : p->slots) {
    if (s.exec) (void)hipGraphExecDestroy(s.exec);
    if (s.done) (void)hipEventDestroy(s.done);
    if (s.stream) (void)hipStreamDestroy(s.stream);
    if (s.h_planes) (void)hipHostFree(s.h_planes);
    if (s.h_legal) (void)hipHostFree(s.h_legal);
    if (s.h_policy) (void)hipHostFree(s.h_policy);
    if (s.h_value) (void)hipHostFree(s.h_value);
    if (s.d_planes) (void)hipFree(s.d_planes);
    if (s.d_legal) (void)hipFree(s.d_legal);
    if (s.d_policy) (void)hipFree(s.d_policy);
    if (s.d_value) (void)hipFree(s.d_value);
  }
  p->slots.clear();
}

// Copy-in, evaluation and copy-out of B positions on the slot's stream.
int enqueue(az_pipeline* p, az_pipeline::Slot& s, int B) {
  const size_t np = (size_t)B * p->in_planes * AZ_SQUARES, nm = (size_t)B * p->n_moves;
  hipError_t e = hipMemcpyAsync(s.d_planes, s.h_planes, np * sizeof(float), hipMemcpyHostToDevice, s.stream);
  if (e == hipSuccess) e = hipMemcpyAsync(s.d_legal, s.h_legal, nm, hipMemcpyHostToDevice, s.stream);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: copy in");
  const int st = az_eval_batch(p->net, s.d_planes, s.d_legal, B, s.d_policy, s.d_value, s.stream);
  if (st != AZ_OK) return st;
  e = hipMemcpyAsync(s.h_policy, s.d_policy, nm * sizeof(float), hipMemcpyDeviceToHost, s.stream);
  if (e == hipSuccess) e = hipMemcpyAsync(s.h_value, s.d_value, (size_t)B * sizeof(float), hipMemcpyDeviceToHost, s.stream);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: copy out");
  return AZ_OK;
}

struct DeviceScope {
  int prev = -1;
  hipError_t err = hipSuccess;
  explicit DeviceScope(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != dev) err = hipSetDevice(dev);
    else if (err == hipSuccess) prev = -1;
  }
  ~DeviceScope() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

}  // namespace

extern "C" {

int az_pipeline_create(az_net* net, int32_t max_batch, int32_t slots, int32_t use_graphs, az_pipeline** out) {
  if (!net || !out) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: NULL argument");
  if (slots < 1 || slots > 64) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: slots must be 1..64");
  const az_layer_spec& sp = az_net_spec(net);
  if (max_batch < 1 || max_batch > sp.max_batch)
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: max_batch must be 1..the handle's max_batch");
  az_pipeline* p = new (std::nothrow) az_pipeline;
  if (!p) return az_fail(AZ_ERR_NOMEM, "az_pipeline_create: host allocation failed");
  p->net = net;
  p->device = az_net_device(net);
  p->max_batch = max_batch;
  p->in_planes = sp.in_planes;
  p->n_moves = sp.policy_planes * AZ_SQUARES;
  p->graphs = use_graphs != 0;
  DeviceScope scope(p->device);
  if (scope.err != hipSuccess) {
    delete p;
    return hip_err(scope.err, "az_pipeline_create: device");
  }
  try {
    p->slots.resize(slots);
  } catch (const std::bad_alloc&) {
    delete p;
    return az_fail(AZ_ERR_NOMEM, "az_pipeline_create: host allocation failed");
  }
  const size_t np = (size_t)max_batch * p->in_planes * AZ_SQUARES, nm = (size_t)max_batch * p->n_moves;
  for (auto& s : p->slots) {
    hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&s.h_planes), np * sizeof(float), hipHostMallocDefault);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&s.h_legal), nm, hipHostMallocDefault);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&s.h_policy), nm * sizeof(float), hipHostMallocDefault);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&s.h_value), (size_t)max_batch * sizeof(float), hipHostMallocDefault);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&s.d_planes), np * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&s.d_legal), nm);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&s.d_policy), nm * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&s.d_value), (size_t)max_batch * sizeof(float));
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&s.stream, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
    if (e != hipSuccess) {
      const int st = hip_err(e, "az_pipeline_create: buffers, streams or events");
      release(p);
      delete p;
      return st;
    }
  }
  *out = p;
  return AZ_OK;
}

int az_pipeline_slot(az_pipeline* p, int32_t slot, float** planes, uint8_t** legal, float** policy, float** value) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_slot: bad slot");
  auto& s = p->slots[slot];
  if (planes) *planes = s.h_planes;
  if (legal) *legal = s.h_legal;
  if (policy) *policy = s.h_policy;
  if (value) *value = s.h_value;
  return AZ_OK;
}

int az_pipeline_submit(az_pipeline* p, int32_t slot, int32_t B) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: bad slot");
  if (B < 0 || B > p->max_batch) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: B out of range");
  auto& s = p->slots[slot];
  if (s.submitted) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: slot already in flight (wait first)");
  DeviceScope scope(p->device);
  if (scope.err != hipSuccess) return hip_err(scope.err, "az_pipeline_submit: device");
  if (B > 0) {
    if (!p->graphs) {
      const int st = enqueue(p, s, B);
      if (st != AZ_OK) return st;
    } else {
      if (!s.exec || s.graph_b != B) {
        if (s.exec) {
          (void)hipGraphExecDestroy(s.exec);
          s.exec = nullptr;
        }
        hipError_t e = hipStreamBeginCapture(s.stream, hipStreamCaptureModeThreadLocal);
        if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: begin capture");
        const int st = enqueue(p, s, B);
        hipGraph_t g = nullptr;
        e = hipStreamEndCapture(s.stream, &g);
        if (st != AZ_OK) {
          if (g) (void)hipGraphDestroy(g);
          return st;
        }
        if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: end capture");
        e = hipGraphInstantiate(&s.exec, g, nullptr, nullptr, 0);
        (void)hipGraphDestroy(g);
        if (e != hipSuccess) {
          s.exec = nullptr;
          return hip_err(e, "az_pipeline_submit: instantiate");
        }
        s.graph_b = B;
      }
      const hipError_t e = hipGraphLaunch(s.exec, s.stream);
      if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: graph launch");
    }
  }
  const hipError_t e = hipEventRecord(s.done, s.stream);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: event");
  s.submitted = true;
  return AZ_OK;
}

int az_pipeline_query(az_pipeline* p, int32_t slot) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_query: bad slot");
  auto& s = p->slots[slot];
  if (!s.submitted) return AZ_OK;
  const hipError_t e = hipEventQuery(s.done);
  if (e == hipErrorNotReady) return 1;
  if (e != hipSuccess) return hip_err(e, "az_pipeline_query");
  s.submitted = false;
  return AZ_OK;
}

int az_pipeline_wait(az_pipeline* p, int32_t slot) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_wait: bad slot");
  auto& s = p->slots[slot];
  if (!s.submitted) return AZ_OK;
  const hipError_t e = hipEventSynchronize(s.done);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_wait");
  s.submitted = false;
  return AZ_OK;
}

void az_pipeline_free(az_pipeline* p) {
  if (!p) return;
  DeviceScope scope(p->device);
  for (auto& s : p->slots)
    if (s.stream) (void)hipStreamSynchronize(s.stream);
  release(p);
  delete p;
}

}  // extern "C"
