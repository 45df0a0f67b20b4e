// Host submission pipeline in front of az_eval_batch.
//
// The paper finds that batching alone does not keep its GPUs busy: host-side
// preparation and submission must overlap GPU execution, through preallocated
// staging buffers, asynchronous copies, completion events and graph replay
// (Section 5.2 "Batching and host-side submission").  A pipeline owns `slots`
// slots on one device; each slot has pinned host buffers (written and read by
// the caller), device buffers and completion events.
//
// Without graphs the pipeline runs three in-order streams shared by all slots:
// copy-in, compute and copy-out.  Submitting a slot enqueues its input copies
// on the copy-in stream, its evaluation on the compute stream (after its
// copies, through an event) and its output copies on the copy-out stream
// (after its evaluation).  Copies therefore run at full link bandwidth in
// submission order while the previous slot evaluates, and evaluations never
// share the chip with each other.  With graphs, each slot captures its steps
// on a stream of its own, once per batch size, and replays that graph.
//
// The dense policy (P*64 floats per position) dominates what crosses PCIe,
// while a search node only needs the probabilities of its legal moves.  With
// AZ_PIPE_COMPACT_POLICY a small kernel gathers, per position, the legal
// cells' probabilities in ascending cell order into max_legal floats and counts
// them, and only that is copied back.
//
// A slot's outputs sit in one block, host and device alike: policy rows, then
// (compact) the legal counts, then the values, each sized for max_batch, so a
// full batch leaves the device in a single copy.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <chrono>
#include <condition_variable>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "az.h"
#include "az_internal.h"

struct az_pipeline {
  struct Slot {
    // pinned host buffers: inputs, and the output block with its three parts
    float* h_planes = nullptr;
    uint8_t* h_legal = nullptr;
    float* h_out = nullptr;
    float* h_policy = nullptr;
    int32_t* h_count = nullptr;
    float* h_value = nullptr;
    // device buffers: inputs, the output block (same layout), and in compact
    // mode the dense policy the evaluation writes before compaction
    float* d_planes = nullptr;
    uint8_t* d_legal = nullptr;
    float* d_out = nullptr;
    float* d_policy = nullptr;
    int32_t* d_count = nullptr;
    float* d_value = nullptr;
    float* d_dense = nullptr;
    hipEvent_t in_done = nullptr, eval_done = nullptr, done = nullptr;
    hipStream_t graph_stream = nullptr;
    hipGraphExec_t exec = nullptr;
    int graph_b = 0;
    int last_b = 0;
    bool submitted = false;
  };
  az_net* net = nullptr;
  int device = 0;
  int max_batch = 0, in_planes = 0, n_moves = 0, max_legal = 0;
  size_t row_floats = 0;  // floats per policy row in the output block: max_legal or n_moves
  bool graphs = false, compact = false;
  hipStream_t s_in = nullptr, s_compute = nullptr, s_out = nullptr;
  std::mutex submit_mu;
  std::vector<Slot> slots;
};

namespace {

constexpr int COMPACT_ROWS_PER_BLOCK = 4;
// mask bytes one wave covers per pass (16 per lane), and passes held in registers
constexpr int COMPACT_PASS = 1024;
constexpr int COMPACT_MAX_PASSES = 6;
static_assert(COMPACT_PASS * COMPACT_MAX_PASSES >= 95 * AZ_SQUARES, "policy rows longer than the register window");

// Bit 7 of each byte of the result is set where the byte of x is non-zero.
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t x) {
  return (((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x) & 0x80808080u;
}

// One wave per position.  All of the row's mask bytes are loaded up front (16
// per lane per pass, every load independent); per pass a wave-wide inclusive
// scan of the lanes' legal counts gives each legal cell its rank, and the cell's
// probability is stored at that rank.  Ranks at or past K are counted but not
// stored; the rest of the row is zero-filled.
__global__ __launch_bounds__(64 * COMPACT_ROWS_PER_BLOCK) void az_compact_policy_kernel(
    const float* __restrict__ policy, const uint8_t* __restrict__ legal, int B, int NM, int K,
    float* __restrict__ out, int32_t* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * COMPACT_ROWS_PER_BLOCK + (threadIdx.x >> 6);
  if (row >= B) return;
  const uint8_t* lg = legal + (size_t)row * NM;
  const float* pr = policy + (size_t)row * NM;
  float* o = out + (size_t)row * K;
  uint4 m[COMPACT_MAX_PASSES];
#pragma unroll
  for (int i = 0; i < COMPACT_MAX_PASSES; ++i) {
    // NM is a multiple of 4 (P*64 cells, or the 1,880 from-to actions), so each
    // 4-byte word of a lane's 16 bytes is either in the row or past its end;
    // words past the end read as zero (not legal)
    const int c = i * COMPACT_PASS + 16 * lane;
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cq = c + 4 * q;
      const uint32_t v = *reinterpret_cast<const uint32_t*>(lg + (cq < NM ? cq : 0));  // clamped, unconditional
      w[q] = cq < NM ? v : 0u;
    }
    m[i] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  int base = 0;
#pragma unroll
  for (int i = 0; i < COMPACT_MAX_PASSES; ++i) {
    if (i * COMPACT_PASS >= NM) break;
    const uint32_t w[4] = {nonzero_bytes(m[i].x), nonzero_bytes(m[i].y), nonzero_bytes(m[i].z),
                           nonzero_bytes(m[i].w)};
    const int n = __popc(w[0]) + __popc(w[1]) + __popc(w[2]) + __popc(w[3]);
    int incl = n;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(incl, d);
      if (lane >= d) incl += t;
    }
    int r = base + incl - n;
    const int c0 = i * COMPACT_PASS + 16 * lane;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t bits = w[q];
      while (bits) {
        const int byte = (__ffs(bits) - 1) >> 3;
        bits &= bits - 1;
        if (r < K) o[r] = pr[c0 + 4 * q + byte];
        ++r;
      }
    }
    base += __shfl(incl, 63);
  }
  for (int j = base + lane; j < K; j += 64) o[j] = 0.0f;
  if (lane == 0) count[row] = base;
}

// ---- allocation-free compact evaluation (az_eval_batch_compact_noalloc)
// The dense policy between the evaluation and the compaction lives in this
// file-scope device array instead of a buffer the library allocates: every
// call on a GPU shares that GPU's copy (calls that overlap on one GPU race).
// In host code `scratch` names a host-side stand-in, never the device memory:
// host code uses the address hipGetSymbolAddress returns for the current
// device, kept per device.
constexpr size_t NOALLOC_FLOATS = (size_t)512 * 95 * AZ_SQUARES;  // 512 positions of the longest policy row
static __device__ __align__(256) float scratch[NOALLOC_FLOATS];
constexpr int NOALLOC_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[NOALLOC_MAX_DEVICES] = {};

// The device address of `scratch` on the current device (looked up once per
// device), or nullptr with the status in *st.
float* scratch_for_current_device(int dev, int* st) {
  if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) {
    *st = az_fail(AZ_ERR_UNSUPPORTED, "az_eval_batch_compact_noalloc: device index past 63");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      *st = az_fail(AZ_ERR_DEVICE, "az_eval_batch_compact_noalloc: hipGetSymbolAddress of the scratch array failed");
      return nullptr;
    }
    g_scratch_ptr[dev] = static_cast<float*>(ptr);
  }
  return g_scratch_ptr[dev];
}

int hip_err(hipError_t e, const char* what) {
  (void)hipGetLastError();
  return az_fail(e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation ? AZ_ERR_NOMEM : AZ_ERR_DEVICE, what);
}

void release(az_pipeline* p) {
  for (auto& s : p->slots) {
    if (s.exec) (void)hipGraphExecDestroy(s.exec);
    if (s.in_done) (void)hipEventDestroy(s.in_done);
    if (s.eval_done) (void)hipEventDestroy(s.eval_done);
    if (s.done) (void)hipEventDestroy(s.done);
    if (s.graph_stream) (void)hipStreamDestroy(s.graph_stream);
    az_host_free(s.h_planes);
    az_host_free(s.h_legal);
    az_host_free(s.h_out);
    az_dev_free(s.d_planes);
    az_dev_free(s.d_legal);
    az_dev_free(s.d_out);
    az_dev_free(s.d_dense);
  }
  p->slots.clear();
  if (p->s_in) (void)hipStreamDestroy(p->s_in);
  if (p->s_compute) (void)hipStreamDestroy(p->s_compute);
  if (p->s_out) (void)hipStreamDestroy(p->s_out);
  p->s_in = p->s_compute = p->s_out = nullptr;
}

// Copy-in, evaluation and output of B positions.  With one stream (graph
// capture) everything is ordered on it; otherwise on the pipeline's three
// streams, joined by the slot's events.
int enqueue(az_pipeline* p, az_pipeline::Slot& s, int B, hipStream_t in, hipStream_t compute, hipStream_t outs) {
  const bool one = in == compute;
  const size_t np = (size_t)B * p->in_planes * AZ_SQUARES, nm = (size_t)B * p->n_moves;
  hipError_t e = hipMemcpyAsync(s.d_planes, s.h_planes, np * sizeof(float), hipMemcpyHostToDevice, in);
  if (e == hipSuccess) e = hipMemcpyAsync(s.d_legal, s.h_legal, nm, hipMemcpyHostToDevice, in);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: copy in");
  if (!one) {
    e = hipEventRecord(s.in_done, in);
    if (e == hipSuccess) e = hipStreamWaitEvent(compute, s.in_done, 0);
    if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: copy-in event");
  }
  const int st = az_eval_batch(p->net, s.d_planes, s.d_legal, B, p->compact ? s.d_dense : s.d_policy, s.d_value,
                               compute);
  if (st != AZ_OK) return st;
  if (p->compact) {
    hipLaunchKernelGGL(az_compact_policy_kernel, dim3((B + COMPACT_ROWS_PER_BLOCK - 1) / COMPACT_ROWS_PER_BLOCK),
                       dim3(64 * COMPACT_ROWS_PER_BLOCK), 0, compute, s.d_dense, s.d_legal, B, p->n_moves,
                       p->max_legal, s.d_policy, s.d_count);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: compaction launch");
  }
  if (!one) {
    e = hipEventRecord(s.eval_done, compute);
    if (e == hipSuccess) e = hipStreamWaitEvent(outs, s.eval_done, 0);
    if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: evaluation event");
  }
  if (B == p->max_batch) {
    // the whole output block in one copy
    const size_t n = (size_t)B * (p->row_floats + 1 + (p->compact ? 1 : 0));
    e = hipMemcpyAsync(s.h_out, s.d_out, n * sizeof(float), hipMemcpyDeviceToHost, outs);
  } else {
    e = hipMemcpyAsync(s.h_policy, s.d_policy, (size_t)B * p->row_floats * sizeof(float), hipMemcpyDeviceToHost, outs);
    if (e == hipSuccess && p->compact)
      e = hipMemcpyAsync(s.h_count, s.d_count, (size_t)B * sizeof(int32_t), hipMemcpyDeviceToHost, outs);
    if (e == hipSuccess)
      e = hipMemcpyAsync(s.h_value, s.d_value, (size_t)B * sizeof(float), hipMemcpyDeviceToHost, outs);
  }
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: copy out");
  return AZ_OK;
}

// After a completed compact submission: every row's legal moves fitted.
int check_counts(const az_pipeline* p, const az_pipeline::Slot& s) {
  if (!p->compact) return AZ_OK;
  for (int r = 0; r < s.last_b; ++r)
    if (s.h_count[r] > p->max_legal) {
      char msg[160];
      snprintf(msg, sizeof msg, "az_pipeline: position %d has %d legal moves, more than max_legal %d (truncated)",
               r, (int)s.h_count[r], p->max_legal);
      return az_fail(AZ_ERR_INVALID_ARG, msg);
    }
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

template <class T>
hipError_t host_alloc(T** ptr, size_t n) {
  return az_host_malloc(reinterpret_cast<void**>(ptr), n * sizeof(T));
}

template <class T>
hipError_t dev_alloc(T** ptr, size_t n) {
  return az_dev_malloc(reinterpret_cast<void**>(ptr), n * sizeof(T));
}

}  // namespace

extern "C" {

int az_pipeline_create(az_net* net, int32_t max_batch, int32_t slots, int32_t flags, int32_t max_legal,
                       az_pipeline** out) {
  if (!net || !out) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: NULL argument");
  if (slots < 1 || slots > 64) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: slots must be 1..64");
  if (flags & ~(AZ_PIPE_GRAPHS | AZ_PIPE_COMPACT_POLICY))
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: unknown flags");
  const bool compact = (flags & AZ_PIPE_COMPACT_POLICY) != 0;
  if (compact ? max_legal < 1 : max_legal != 0)
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: max_legal must be >= 1 with AZ_PIPE_COMPACT_POLICY, else 0");
  const az_layer_spec& sp = az_net_spec(net);
  if (max_batch < 1 || max_batch > sp.max_batch)
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: max_batch must be 1..the handle's max_batch");
  if (compact && max_legal > az_spec_moves(sp))
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_create: max_legal exceeds the number of policy cells");
  if (az_spec_moves(sp) > COMPACT_PASS * COMPACT_MAX_PASSES)
    return az_fail(AZ_ERR_UNSUPPORTED, "az_pipeline_create: policy rows too long");
  az_pipeline* p = new (std::nothrow) az_pipeline;
  if (!p) return az_fail(AZ_ERR_NOMEM, "az_pipeline_create: host allocation failed");
  p->net = net;
  p->device = az_net_device(net);
  p->max_batch = max_batch;
  p->in_planes = sp.in_planes;
  p->n_moves = az_spec_moves(sp);
  p->graphs = (flags & AZ_PIPE_GRAPHS) != 0;
  p->compact = compact;
  p->max_legal = max_legal;
  p->row_floats = compact ? (size_t)max_legal : (size_t)p->n_moves;
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
  // output block: policy rows, legal counts (compact), values
  const size_t n_out = (size_t)max_batch * (p->row_floats + 1 + (compact ? 1 : 0));
  hipError_t e = hipSuccess;
  if (!p->graphs) {
    e = hipStreamCreateWithFlags(&p->s_in, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->s_compute, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->s_out, hipStreamNonBlocking);
  }
  for (auto& s : p->slots) {
    if (e != hipSuccess) break;
    e = host_alloc(&s.h_planes, np);
    if (e == hipSuccess) e = host_alloc(&s.h_legal, nm);
    if (e == hipSuccess) e = host_alloc(&s.h_out, n_out);
    if (e == hipSuccess) e = dev_alloc(&s.d_planes, np);
    if (e == hipSuccess) e = dev_alloc(&s.d_legal, nm);
    if (e == hipSuccess) e = dev_alloc(&s.d_out, n_out);
    if (e == hipSuccess && compact) e = dev_alloc(&s.d_dense, nm);
    if (e == hipSuccess) {
      const size_t nv = (size_t)max_batch * p->row_floats;
      s.h_policy = s.h_out;
      s.d_policy = s.d_out;
      if (compact) {
        s.h_count = reinterpret_cast<int32_t*>(s.h_out + nv);
        s.d_count = reinterpret_cast<int32_t*>(s.d_out + nv);
      }
      s.h_value = s.h_out + nv + (compact ? max_batch : 0);
      s.d_value = s.d_out + nv + (compact ? max_batch : 0);
    }
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.in_done, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.eval_done, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
    if (e == hipSuccess && p->graphs) e = hipStreamCreateWithFlags(&s.graph_stream, hipStreamNonBlocking);
  }
  if (e != hipSuccess) {
    const int st = hip_err(e, "az_pipeline_create: buffers, streams or events");
    release(p);
    delete p;
    return st;
  }
  *out = p;
  return AZ_OK;
}

int az_pipeline_slot(az_pipeline* p, int32_t slot, float** planes, uint8_t** legal, float** policy, float** value,
                     int32_t** legal_count) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_slot: bad slot");
  auto& s = p->slots[slot];
  if (planes) *planes = s.h_planes;
  if (legal) *legal = s.h_legal;
  if (policy) *policy = s.h_policy;
  if (value) *value = s.h_value;
  if (legal_count) *legal_count = s.h_count;
  return AZ_OK;
}

int az_pipeline_submit(az_pipeline* p, int32_t slot, int32_t B) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: bad slot");
  if (B < 0 || B > p->max_batch) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: B out of range");
  auto& s = p->slots[slot];
  if (s.submitted) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_submit: slot already in flight (wait first)");
  DeviceScope scope(p->device);
  if (scope.err != hipSuccess) return hip_err(scope.err, "az_pipeline_submit: device");
  hipError_t e = hipSuccess;
  if (!p->graphs) {
    // the shared streams take the slots' work in submission order
    std::lock_guard<std::mutex> lock(p->submit_mu);
    if (B > 0) {
      const int st = enqueue(p, s, B, p->s_in, p->s_compute, p->s_out);
      if (st != AZ_OK) return st;
    }
    e = hipEventRecord(s.done, p->s_out);
  } else {
    if (B > 0) {
      if (!s.exec || s.graph_b != B) {
        if (s.exec) {
          (void)hipGraphExecDestroy(s.exec);
          s.exec = nullptr;
        }
        e = hipStreamBeginCapture(s.graph_stream, hipStreamCaptureModeThreadLocal);
        if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: begin capture");
        const int st = enqueue(p, s, B, s.graph_stream, s.graph_stream, s.graph_stream);
        hipGraph_t g = nullptr;
        e = hipStreamEndCapture(s.graph_stream, &g);
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
      e = hipGraphLaunch(s.exec, s.graph_stream);
      if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: graph launch");
    }
    e = hipEventRecord(s.done, s.graph_stream);
  }
  if (e != hipSuccess) return hip_err(e, "az_pipeline_submit: event");
  s.submitted = true;
  s.last_b = B;
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
  return check_counts(p, s);
}

int az_pipeline_wait(az_pipeline* p, int32_t slot) {
  if (!p || slot < 0 || slot >= (int)p->slots.size()) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_wait: bad slot");
  auto& s = p->slots[slot];
  if (!s.submitted) return AZ_OK;
  const hipError_t e = hipEventSynchronize(s.done);
  if (e != hipSuccess) return hip_err(e, "az_pipeline_wait");
  s.submitted = false;
  return check_counts(p, s);
}

int az_pipeline_drive(az_pipeline* p, int32_t workers, int32_t slots_per_worker, int32_t B, int32_t warmup,
                      int32_t batches, double* seconds) {
  if (!p || !seconds) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_drive: NULL argument");
  if (workers < 1 || slots_per_worker < 1 || (int64_t)workers * slots_per_worker > (int64_t)p->slots.size())
    return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_drive: workers x slots_per_worker exceeds the pipeline's slots");
  if (B < 1 || B > p->max_batch) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_drive: B out of range");
  if (warmup < 0 || batches < 1) return az_fail(AZ_ERR_INVALID_ARG, "az_pipeline_drive: bad batch counts");
  // A barrier between the warm-up and the timed part: the main thread starts
  // the clock once every worker has drained its warm-up submissions.
  // Error messages are per thread: a worker's is copied out and set again on
  // the calling thread.
  std::mutex mu;
  std::condition_variable cv;
  int arrived = 0;
  bool go = false, abandon = false;
  std::vector<int> status(workers, AZ_OK);
  std::vector<std::string> message(workers);
  auto run = [&](int w) {
    const int s0 = w * slots_per_worker;
    auto phase = [&](int count) {
      for (int i = 0; i < count; ++i) {
        const int k = s0 + i % slots_per_worker;
        int st = az_pipeline_wait(p, k);
        if (st == AZ_OK) st = az_pipeline_submit(p, k, B);
        if (st != AZ_OK) return st;
      }
      for (int k = s0; k < s0 + slots_per_worker; ++k) {
        const int st = az_pipeline_wait(p, k);
        if (st != AZ_OK) return st;
      }
      return (int)AZ_OK;
    };
    int st = phase(warmup);
    {
      std::unique_lock<std::mutex> lock(mu);
      ++arrived;
      cv.notify_all();
      cv.wait(lock, [&] { return go; });
    }
    if (st == AZ_OK && !abandon) st = phase(batches);
    status[w] = st;
    if (st != AZ_OK) message[w] = az_last_error();
  };
  std::vector<std::thread> th;
  try {
    for (int w = 0; w < workers; ++w) th.emplace_back(run, w);
  } catch (...) {
    {
      std::lock_guard<std::mutex> lock(mu);
      go = abandon = true;
    }
    cv.notify_all();
    for (auto& t : th) t.join();
    return az_fail(AZ_ERR_NOMEM, "az_pipeline_drive: could not start the worker threads");
  }
  {
    std::unique_lock<std::mutex> lock(mu);
    cv.wait(lock, [&] { return arrived == workers; });
    go = true;
  }
  const auto t0 = std::chrono::steady_clock::now();
  cv.notify_all();
  for (auto& t : th) t.join();
  *seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  for (int w = 0; w < workers; ++w)
    if (status[w] != AZ_OK) return az_fail(status[w], message[w].c_str());
  return AZ_OK;
}

int az_eval_batch_compact_noalloc(az_net* net, const float* planes, const uint8_t* legal, int32_t B,
                                  int32_t max_legal, float* policy, int32_t* legal_count, float* value,
                                  void* stream) {
  if (!net) return az_fail(AZ_ERR_INVALID_ARG, "az_eval_batch_compact_noalloc: NULL handle");
  const az_layer_spec& sp = az_net_spec(net);
  const int nm = az_spec_moves(sp);
  if (max_legal < 1 || max_legal > nm)
    return az_fail(AZ_ERR_INVALID_ARG, "az_eval_batch_compact_noalloc: max_legal must be 1..az_net_moves(net)");
  if (B < 0 || B > sp.max_batch) return az_fail(AZ_ERR_INVALID_ARG, "az_eval_batch_compact_noalloc: B out of range");
  if ((size_t)B * (size_t)nm > NOALLOC_FLOATS) {
    char msg[200];
    snprintf(msg, sizeof msg,
             "az_eval_batch_compact_noalloc: B = %d needs %zu floats of scratch, more than its %zu (at most %zu positions "
             "of %d policy cells)",
             (int)B, (size_t)B * (size_t)nm, NOALLOC_FLOATS, NOALLOC_FLOATS / (size_t)nm, nm);
    return az_fail(AZ_ERR_INVALID_ARG, msg);
  }
  if (B == 0) return AZ_OK;
  if (!planes || !legal || !policy || !legal_count || !value)
    return az_fail(AZ_ERR_INVALID_ARG, "az_eval_batch_compact_noalloc: NULL buffer");
  if (((uintptr_t)policy | (uintptr_t)legal_count) & 3u)
    return az_fail(AZ_ERR_INVALID_ARG, "az_eval_batch_compact_noalloc: policy and legal_count must be 4-byte aligned");
  DeviceScope scope(az_net_device(net));
  if (scope.err != hipSuccess) return hip_err(scope.err, "az_eval_batch_compact_noalloc: device");
  int st = AZ_OK;
  float* dense = scratch_for_current_device(az_net_device(net), &st);
  if (!dense) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = az_eval_batch(net, planes, legal, B, dense, value, s);
  if (st != AZ_OK) return st;
  hipLaunchKernelGGL(az_compact_policy_kernel, dim3((B + COMPACT_ROWS_PER_BLOCK - 1) / COMPACT_ROWS_PER_BLOCK),
                     dim3(64 * COMPACT_ROWS_PER_BLOCK), 0, s, dense, legal, B, nm, max_legal, policy, legal_count);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_err(e, "az_eval_batch_compact_noalloc: compaction launch");
  return AZ_OK;
}

void az_pipeline_free(az_pipeline* p) {
  if (!p) return;
  DeviceScope scope(p->device);
  for (auto& s : p->slots)
    if (s.graph_stream) (void)hipStreamSynchronize(s.graph_stream);
  for (hipStream_t st : {p->s_in, p->s_compute, p->s_out})
    if (st) (void)hipStreamSynchronize(st);
  release(p);
  delete p;
}

}  // extern "C"
