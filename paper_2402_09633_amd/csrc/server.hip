// Request queue for serving one model to many callers on one GPU: the
// single-GPU form of the inference service of paper sections 2.3 and 3.2,
// where one GPU runs several instances of the model (Fig. 4b) and requests
// from many clients queue in front of them.
//
// n_instances worker threads each own one HIP stream (default priority) and
// take requests from one FIFO queue; every request is one gnn_infer call on
// the shared handle (the library is reentrant across streams), followed by a
// synchronisation of the worker's stream.  Latency is measured on the host
// from submission to completion, so it includes the time spent queued.  Each
// request is also bracketed by two events on the worker's stream, which give
// its device interval relative to an event recorded when the server was
// created: the union of those intervals over a run is the time the GPU spent
// on requests (the utilisation of the paper's Fig. 4b).
#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <deque>
#include <mutex>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "../../include/gnn.h"
#include "gnn_internal.h"

namespace {

using clock_t_ = std::chrono::steady_clock;

struct Request {
  const float *x = nullptr;
  const int32_t *ei = nullptr;
  int64_t n_nodes = 0, n_edges = 0;
  float *out = nullptr;
  clock_t_::time_point submitted, done_at;
  double dev_start_ms = -1.0, dev_end_ms = -1.0;  // device interval (< 0: unknown)
  bool done = false;
  bool claimed = false;  // a thread is waiting for it (only that one may release it)
  int status = GNN_OK;
  std::string error;
};

}  // namespace

struct gnn_server {
  gnn_handle *model = nullptr;
  int device = 0;
  std::vector<std::thread> workers;
  std::mutex mu;
  std::condition_variable cv_work, cv_done;
  std::deque<int64_t> queue;
  // Node-based map: references to its elements stay valid when a submit
  // rehashes it; only the claiming waiter erases an element.
  std::unordered_map<int64_t, Request> reqs;
  int64_t next_id = 0;
  bool stopping = false;
  int start_errors = 0;
  hipEvent_t t0 = nullptr;  // time origin of the device intervals
};

namespace {

void worker(gnn_server *s) {
  hipStream_t stream = nullptr;
  hipEvent_t ev[2] = {nullptr, nullptr};
  const bool ok = hipSetDevice(s->device) == hipSuccess &&
                  hipStreamCreateWithFlags(&stream, hipStreamNonBlocking) == hipSuccess &&
                  hipEventCreate(&ev[0]) == hipSuccess && hipEventCreate(&ev[1]) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
    if (stream) (void)hipStreamDestroy(stream);
    std::lock_guard<std::mutex> lk(s->mu);
    ++s->start_errors;
    s->cv_done.notify_all();
    return;
  }
  for (;;) {
    int64_t id;
    Request r;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv_work.wait(lk, [&] { return s->stopping || !s->queue.empty(); });
      if (s->queue.empty()) break;  // stopping and drained
      id = s->queue.front();
      s->queue.pop_front();
      r = s->reqs.at(id);
    }
    // (the events are reused: the previous request's work has finished)
    const bool timed = hipEventRecord(ev[0], stream) == hipSuccess;
    if (!timed) (void)hipGetLastError();
    int rc = gnn_infer(s->model, r.x, r.ei, r.n_nodes, r.n_edges, r.out, stream);
    const bool timed_end = timed && hipEventRecord(ev[1], stream) == hipSuccess;
    std::string err;
    if (rc == GNN_OK) {
      const hipError_t e = hipStreamSynchronize(stream);
      if (e != hipSuccess) {
        rc = GNN_E_HIP;
        err = std::string("stream synchronisation failed: ") + hipGetErrorString(e);
      }
    } else {
      err = gnn_last_error();
    }
    float t_a = -1.f, t_b = -1.f;
    if (!(rc == GNN_OK && timed_end && hipEventSynchronize(ev[1]) == hipSuccess &&
          hipEventElapsedTime(&t_a, s->t0, ev[0]) == hipSuccess &&
          hipEventElapsedTime(&t_b, s->t0, ev[1]) == hipSuccess)) {
      (void)hipGetLastError();
      t_a = t_b = -1.f;
    }
    {
      std::lock_guard<std::mutex> lk(s->mu);
      Request &q = s->reqs.at(id);
      q.status = rc;
      q.error = err;
      q.done_at = clock_t_::now();
      q.dev_start_ms = t_a;
      q.dev_end_ms = t_b;
      q.done = true;
    }
    s->cv_done.notify_all();
  }
  // the handle's cached workspaces must not keep events of this stream
  (void)hipStreamSynchronize(stream);
  gnn::ws_forget_stream(s->model, stream);
  for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  (void)hipStreamDestroy(stream);
  (void)hipGetLastError();
}

// Waits for request `id`, releases it and returns a copy.  Only one thread
// may wait for a given request: a second one gets GNN_E_INVALID_ARG.
int take_request(gnn_server *s, int64_t id, Request *out) {
  if (!s) return gnn::set_error(GNN_E_INVALID_ARG, "server is NULL");
  std::unique_lock<std::mutex> lk(s->mu);
  {
    auto it = s->reqs.find(id);
    if (it == s->reqs.end()) return gnn::set_error(GNN_E_INVALID_ARG, "unknown request id");
    if (it->second.claimed)
      return gnn::set_error(GNN_E_INVALID_ARG, "another thread is waiting for this request");
    it->second.claimed = true;
  }
  // Looked up again after every wake-up: a submit may have rehashed the map.
  s->cv_done.wait(lk, [&] {
    return s->reqs.at(id).done || s->start_errors == (int)s->workers.size();
  });
  auto it = s->reqs.find(id);
  if (!it->second.done) {
    it->second.claimed = false;
    return gnn::set_error(GNN_E_HIP, "no worker could create its stream");
  }
  *out = it->second;
  s->reqs.erase(it);
  return GNN_OK;
}

}  // namespace

extern "C" {

gnn_server *gnn_server_create(gnn_handle *h, int n_instances) {
  if (!h || n_instances < 1 || n_instances > 64) {
    gnn::set_error(GNN_E_INVALID_ARG, h ? "n_instances outside 1..64" : "handle is NULL");
    return nullptr;
  }
  gnn_server *s = new gnn_server();
  s->model = h;
  if (hipGetDevice(&s->device) != hipSuccess) {
    delete s;
    gnn::set_error(GNN_E_NO_DEVICE, "hipGetDevice failed");
    return nullptr;
  }
  if (hipEventCreate(&s->t0) != hipSuccess || hipEventRecord(s->t0, nullptr) != hipSuccess ||
      hipEventSynchronize(s->t0) != hipSuccess) {
    (void)hipGetLastError();
    if (s->t0) (void)hipEventDestroy(s->t0);
    delete s;
    gnn::set_error(GNN_E_HIP, "creating the server's time-origin event failed");
    return nullptr;
  }
  for (int i = 0; i < n_instances; ++i) s->workers.emplace_back(worker, s);
  return s;
}

int64_t gnn_server_submit(gnn_server *s, const float *node_feat, const int32_t *edge_index,
                          int64_t n_nodes, int64_t n_edges, float *edge_scores) {
  if (!s) return gnn::set_error(GNN_E_INVALID_ARG, "server is NULL");
  if (!node_feat || !edge_index || !edge_scores)
    return gnn::set_error(GNN_E_INVALID_ARG, "NULL input or output pointer");
  if (n_nodes < 0 || n_edges < 0 || n_nodes > INT32_MAX || n_edges > INT32_MAX)
    return gnn::set_error(GNN_E_INVALID_ARG, "count outside 0..INT32_MAX");
  std::lock_guard<std::mutex> lk(s->mu);
  if (s->stopping) return gnn::set_error(GNN_E_INVALID_ARG, "server is shutting down");
  if (s->start_errors == (int)s->workers.size())
    return gnn::set_error(GNN_E_HIP, "no worker could create its stream");
  const int64_t id = s->next_id++;
  Request &r = s->reqs[id];
  r.x = node_feat;
  r.ei = edge_index;
  r.n_nodes = n_nodes;
  r.n_edges = n_edges;
  r.out = edge_scores;
  r.submitted = clock_t_::now();
  s->queue.push_back(id);
  s->cv_work.notify_one();
  return id;
}

int gnn_server_wait(gnn_server *s, int64_t id, double *latency_ms) {
  Request r;
  const int rc = take_request(s, id, &r);
  if (rc != GNN_OK) return rc;
  if (latency_ms)
    *latency_ms = std::chrono::duration<double, std::milli>(r.done_at - r.submitted).count();
  if (r.status != GNN_OK) return gnn::set_error(r.status, r.error.c_str());
  return GNN_OK;
}

int gnn_server_wait_info(gnn_server *s, int64_t id, gnn_request_info *info) {
  if (!info || info->struct_size != sizeof(gnn_request_info))
    return gnn::set_error(GNN_E_INVALID_ARG, "info is NULL or info->struct_size is wrong");
  Request r;
  const int rc = take_request(s, id, &r);
  if (rc != GNN_OK) return rc;
  info->status = r.status;
  info->latency_ms = std::chrono::duration<double, std::milli>(r.done_at - r.submitted).count();
  info->device_start_ms = r.dev_start_ms;
  info->device_end_ms = r.dev_end_ms;
  if (r.status != GNN_OK) return gnn::set_error(r.status, r.error.c_str());
  return GNN_OK;
}

void gnn_server_destroy(gnn_server *s) {
  if (!s) return;
  {
    std::lock_guard<std::mutex> lk(s->mu);
    s->stopping = true;
  }
  s->cv_work.notify_all();
  for (auto &t : s->workers) t.join();
  (void)hipEventDestroy(s->t0);
  delete s;
}

}  // extern "C"
