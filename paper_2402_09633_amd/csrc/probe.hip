// Streaming-rate probe: the HBM read, write and copy rates that plain,
// fully coalesced kernels reach on this device.  They are the achievable
// ceilings beside the 8 TB/s peak against which the inference kernels'
// bandwidth is reported (a kernel that reads R bytes and writes W bytes
// cannot finish faster than R / read_rate + W / write_rate).  Not part of
// the method; only measurement uses it.
#include <cstdio>

#include "../../include/gnn.h"
#include "gnn_internal.h"

namespace gnn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int PROBE_THREADS = 256;

// Every element is read once; the sum is stored only if it equals a value
// that zero-filled or finite data cannot produce, so the loads stay.
__global__ __launch_bounds__(PROBE_THREADS) void probe_read(const f4 *__restrict__ a, int64_t n,
                                                            float *__restrict__ sink) {
  f4 s = {0.f, 0.f, 0.f, 0.f};
  for (int64_t i = (int64_t)blockIdx.x * PROBE_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * PROBE_THREADS)
    s += __builtin_nontemporal_load(a + i);
  const float t = s[0] + s[1] + s[2] + s[3];
  if (t == -1.5e38f) sink[0] = t;
}

__global__ __launch_bounds__(PROBE_THREADS) void probe_write(f4 *__restrict__ a, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * PROBE_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * PROBE_THREADS)
    __builtin_nontemporal_store(f4{1.f, 2.f, 3.f, 4.f}, a + i);
}

__global__ __launch_bounds__(PROBE_THREADS) void probe_copy(const f4 *__restrict__ a,
                                                            f4 *__restrict__ b, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * PROBE_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * PROBE_THREADS)
    __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

hipError_t launch_probe(int kind, void *buf, void *buf2, int64_t n, int grid, hipStream_t st) {
  if (kind == GNN_PROBE_READ)
    probe_read<<<grid, PROBE_THREADS, 0, st>>>((const f4 *)buf, n, (float *)buf2);
  else if (kind == GNN_PROBE_WRITE)
    probe_write<<<grid, PROBE_THREADS, 0, st>>>((f4 *)buf, n);
  else
    probe_copy<<<grid, PROBE_THREADS, 0, st>>>((const f4 *)buf, (f4 *)buf2, n);
  return hipGetLastError();
}

}  // namespace
}  // namespace gnn

extern "C" int gnn_hbm_probe(int kind, void *buf, void *buf2, int64_t bytes, int32_t grid,
                             int32_t reps, float *ms, hipStream_t stream) {
  using gnn::set_error;
  if (!ms) return set_error(GNN_E_INVALID_ARG, "ms is NULL");
  *ms = 0.f;
  if (kind != GNN_PROBE_READ && kind != GNN_PROBE_WRITE && kind != GNN_PROBE_COPY)
    return set_error(GNN_E_INVALID_ARG, "kind is not GNN_PROBE_READ, _WRITE or _COPY");
  if (bytes <= 0 || bytes % 16) return set_error(GNN_E_INVALID_ARG, "bytes must be a positive multiple of 16");
  if (!buf || !buf2) return set_error(GNN_E_INVALID_ARG, "buf or buf2 is NULL");
  if (grid < 0 || reps < 1 || reps > 1000)
    return set_error(GNN_E_INVALID_ARG, "grid must be >= 0 and reps in 1..1000");
  int dev = 0, n_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    return set_error(GNN_E_NO_DEVICE, "no current HIP device");
  }
  const int g = grid > 0 ? grid : 4 * n_cu;
  const int64_t n = bytes / 16;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    (void)hipGetLastError();
    return set_error(GNN_E_HIP, "hipEventCreate failed");
  }
  int rc = GNN_OK;
  float best = 0.f;
  hipError_t e = gnn::launch_probe(kind, buf, buf2, n, g, stream);  // warm-up
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    e = hipEventRecord(e0, stream);
    if (e == hipSuccess) e = gnn::launch_probe(kind, buf, buf2, n, g, stream);
    if (e == hipSuccess) e = hipEventRecord(e1, stream);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
    if (e == hipSuccess && (r == 0 || t < best)) best = t;
  }
  if (e != hipSuccess) {
    char msg[160];
    snprintf(msg, sizeof msg, "probe launch failed: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    rc = set_error(GNN_E_HIP, msg);
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (rc == GNN_OK) *ms = best;
  return rc;
}
