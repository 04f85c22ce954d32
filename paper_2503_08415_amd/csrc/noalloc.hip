// noalloc.hip -- ts_sweep_run_static: a whole sweep in one call that
// allocates no device memory.  Every buffer the kernels use (traces, units,
// work order, ticket counters, preempted queues, latency arrays, results,
// per-request records, the disaggregated points' stage buffers) is carved
// out of one file-scope device array of
// TS_STATIC_SCRATCH_BYTES, which each GPU the library runs on holds until
// the process ends.  The kernels and the launch sequence are those of
// ts_sweep_create + ts_sweep_run.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <mutex>

#include "sweep_host.h"

namespace {

constexpr size_t kScratchBytes = TS_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

// The scratch.  Host code never passes this name to a kernel or a copy (on
// the host it is only a stand-in for the symbol): it uses the device address
// that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;                              // set-up and calls, one at a time
unsigned char* g_scratch_ptr[kMaxDevices] = {};  // device address of scratch, per device

// The device address of this device's scratch, looked up once per device
// with that device current.
int scratch_of(int dev, unsigned char** out) {
  if (dev < 0 || dev >= kMaxDevices) {
    tsw::set_error_text("device index beyond the static scratch table");
    return TS_ERR_UNSUPPORTED;
  }
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return tsw::device_error(e, "hipGetSymbolAddress(scratch)");
    if (!p) {
      tsw::set_error_text("hipGetSymbolAddress(scratch) returned no address");
      return TS_ERR_DEVICE;
    }
    g_scratch_ptr[dev] = (unsigned char*)p;
  }
  *out = g_scratch_ptr[dev];
  return TS_OK;
}

// Lays the buffers out one after another, each aligned to 256 bytes.
struct Carver {
  unsigned char* base;
  size_t used = 0;
  template <typename T>
  T* take(size_t count) {
    used = (used + 255) & ~(size_t)255;
    T* p = reinterpret_cast<T*>(base + used);
    used += std::max<size_t>(count, 1) * sizeof(T);
    return p;
  }
};

// Fills B from the scratch at base (or only measures when base is null);
// returns the bytes used.
size_t carve(const tsw::Plan& P, unsigned char* base, tsw::DevBufs* B) {
  const tsw::BufCounts n = tsw::buf_counts(P);
  Carver c{base};
  tsw::DevBufs b;
  b.recs = c.take<tsw::TraceRec>(n.recs);
  b.points = c.take<tsw::DevPoint>(n.points);
  b.order = c.take<int32_t>(n.order);
  b.counter = c.take<unsigned int>(n.counter);
  b.queue = c.take<tsw::QEntry>(n.queue);
  b.res = c.take<ts_point_result>(n.res);
  b.e2e = c.take<int64_t>(n.lat);
  b.ttft = c.take<int64_t>(n.lat);
  b.req = c.take<ts_req_result>(n.req);
  b.pd = c.take<tsw::PdAux>(n.pd);
  b.s1_admit = c.take<int64_t>(n.s1);
  b.s1_first = c.take<int64_t>(n.s1);
  b.sub_a2 = c.take<int64_t>(n.sub);
  b.sub_gid = c.take<int32_t>(n.sub);
  b.gids = c.take<int32_t>(n.gids);
  b.pinfo = c.take<tsw::PointInfo>(n.pinfo);
  b.handed = c.take<int32_t>(n.handed);
  b.work = c.take<unsigned long long>(n.work);
  b.resume = c.take<unsigned char>(n.resume * tsw::kResumeBytes);
  b.claim = c.take<unsigned int>(n.claim);
  if (B) *B = b;
  return c.used;
}

}  // namespace

extern "C" int ts_sweep_run_static(const ts_model* model, const ts_trace* traces,
                                   int32_t n_traces, const ts_point* points, int32_t n_points,
                                   const ts_options* opt, void* hip_stream,
                                   ts_point_result* out_points, ts_req_result* out_requests) {
  tsw::clear_error_text();
  std::lock_guard<std::mutex> lock(g_mu);
  tsw::Plan P;
  int rc = tsw::make_plan(model, traces, n_traces, points, n_points, opt, &P);
  if (rc != TS_OK) return rc;
  if (!out_points && P.count > 0) return TS_ERR_ARG;
  if (out_requests && !(P.flags & TS_F_PER_REQUEST)) return TS_ERR_STATE;
  if ((P.flags & TS_F_PER_REQUEST) && !out_requests && P.count > 0) return TS_ERR_ARG;
  // The per-workgroup queues scale with the grid: shrink it until
  // everything fits, down to one workgroup per launch.
  while (carve(P, nullptr, nullptr) > kScratchBytes && P.max_grid() > 1) {
    const int g = std::max(1, P.max_grid() / 2);
    for (int l = 0; l < tsw::kLaunches; ++l) P.grid[l] = std::min(P.grid[l], g);
  }
  const size_t need = carve(P, nullptr, nullptr);
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof msg, "the sweep needs %zu bytes of device memory; the static scratch "
             "holds %zu", need, kScratchBytes);
    tsw::set_error_text(msg);
    return TS_ERR_UNSUPPORTED;
  }
  hipError_t e = hipSetDevice(P.device);
  if (e != hipSuccess) return tsw::device_error(e, "hipSetDevice");
  unsigned char* base = nullptr;
  rc = scratch_of(P.device, &base);
  if (rc != TS_OK) return rc;
  tsw::DevBufs B;
  carve(P, base, &B);
  hipStream_t s = (hipStream_t)hip_stream;
  // inputs from the plan's host vectors, which live until the stream is
  // synchronised below; the enqueue clears the ticket counters, and every
  // request record is rewritten by the run
  rc = tsw::upload(P, B, true, s);
  if (rc == TS_OK) rc = tsw::enqueue(P, B, s, nullptr);
  if (rc == TS_OK && P.count > 0) {
    e = hipMemcpyAsync(out_points, B.res, (size_t)P.count * sizeof(ts_point_result),
                       hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && out_requests)
      e = hipMemcpyAsync(out_requests, B.req,
                         (size_t)P.count * (size_t)P.max_n * sizeof(ts_req_result),
                         hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) rc = tsw::device_error(e, "copy results");
  }
  // always drain the stream before the host vectors go out of scope
  e = hipStreamSynchronize(s);
  if (rc == TS_OK && e != hipSuccess) rc = tsw::device_error(e, "stream synchronize");
  return rc;
}
