// Request queue for serving one model to many callers on one GPU: the
// single-GPU form of the inference service of paper sections 2.3 and 3.2,
// where one GPU runs several instances of the model (Fig. 4b) and requests
// from many clients queue in front of them.
//
// n_instances worker threads each own one HIP stream (default priority) and
// take requests from one FIFO queue; every request is one gnn_infer call on
// the shared handle (the library is reentrant across streams), followed by a
// synchronisation of the worker's stream.  Latency is measured on the host
// from submission to completion, so it includes the time spent queued.
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
  bool done = false;
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
  std::unordered_map<int64_t, Request> reqs;
  int64_t next_id = 0;
  bool stopping = false;
  int start_errors = 0;
};

namespace {

void worker(gnn_server *s) {
  hipStream_t stream = nullptr;
  const bool ok = hipSetDevice(s->device) == hipSuccess &&
                  hipStreamCreateWithFlags(&stream, hipStreamNonBlocking) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
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
      r = s->reqs[id];
    }
    int rc = gnn_infer(s->model, r.x, r.ei, r.n_nodes, r.n_edges, r.out, stream);
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
    {
      std::lock_guard<std::mutex> lk(s->mu);
      Request &q = s->reqs[id];
      q.status = rc;
      q.error = err;
      q.done_at = clock_t_::now();
      q.done = true;
    }
    s->cv_done.notify_all();
  }
  (void)hipStreamDestroy(stream);
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
  if (!s) return gnn::set_error(GNN_E_INVALID_ARG, "server is NULL");
  std::unique_lock<std::mutex> lk(s->mu);
  auto it = s->reqs.find(id);
  if (it == s->reqs.end()) return gnn::set_error(GNN_E_INVALID_ARG, "unknown request id");
  s->cv_done.wait(lk, [&] {
    return it->second.done || s->start_errors == (int)s->workers.size();
  });
  if (!it->second.done) return gnn::set_error(GNN_E_HIP, "no worker could create its stream");
  const Request r = it->second;
  s->reqs.erase(it);
  lk.unlock();
  if (latency_ms)
    *latency_ms = std::chrono::duration<double, std::milli>(r.done_at - r.submitted).count();
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
  delete s;
}

}  // extern "C"
