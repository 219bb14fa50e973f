// Open-loop trace replay (tp_run_trace): the calling thread issues requests at their
// arrival times; a completion thread waits for each request's event in issue order.
#include <hip/hip_runtime_api.h>

#include <chrono>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>

#include "../core/errors.hpp"
#include "runtime.hpp"

using namespace tp;

namespace {

constexpr uint32_t kRing = 256;

uint64_t since(std::chrono::steady_clock::time_point t0) {
  return (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0)
      .count();
}

}  // namespace

extern "C" tp_status tp_run_trace(tp_ctx* c, const tp_request* reqs, uint32_t n, void* stream_,
                                  tp_request_result* out) {
  if (!c || (n && (!reqs || !out))) return fail(TP_E_INVAL, "tp_run_trace: NULL argument");
  for (uint32_t i = 1; i < n; ++i)
    if (reqs[i].arrival_ns < reqs[i - 1].arrival_ns) return fail(TP_E_INVAL, "tp_run_trace: arrivals must not decrease");
  if (c->trace_ev.empty()) {
    c->trace_ev.assign(kRing, nullptr);
    for (auto& e : c->trace_ev) {
      hipError_t err = hipEventCreateWithFlags(&e, hipEventDisableTiming);
      if (err != hipSuccess) {
        for (auto& x : c->trace_ev)
          if (x) (void)hipEventDestroy(x);
        c->trace_ev.clear();
        return fail(TP_E_HIP, std::string("tp_run_trace: event creation: ") + hipGetErrorString(err));
      }
    }
  }
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  std::mutex mu;
  std::condition_variable cv;
  std::deque<uint32_t> pending;     // issued requests awaiting completion, in issue order
  uint32_t in_flight = 0;
  bool finished = false;
  hipError_t sync_err = hipSuccess;
  const auto t0 = std::chrono::steady_clock::now();

  std::thread waiter([&] {
    for (;;) {
      uint32_t i;
      {
        std::unique_lock<std::mutex> lk(mu);
        cv.wait(lk, [&] { return !pending.empty() || finished; });
        if (pending.empty()) return;
        i = pending.front();
        pending.pop_front();
      }
      hipError_t e = hipEventSynchronize(c->trace_ev[i % kRing]);
      const uint64_t t = since(t0);
      std::lock_guard<std::mutex> lk(mu);
      out[i].done_ns = t;
      if (e != hipSuccess && sync_err == hipSuccess) sync_err = e;
      --in_flight;
      cv.notify_all();
    }
  });

  tp_status first_err = TP_OK;
  std::string first_msg;
  for (uint32_t i = 0; i < n; ++i) {
    std::this_thread::sleep_until(t0 + std::chrono::nanoseconds(reqs[i].arrival_ns));
    {
      std::unique_lock<std::mutex> lk(mu);
      cv.wait(lk, [&] { return in_flight < kRing; });
    }
    int32_t res = 0;
    (void)tp_is_resident(c, reqs[i].model_id, &res);
    out[i].hit = res;
    out[i].issue_ns = since(t0);
    tp_status st = tp_infer(c, reqs[i].model_id, reqs[i].input_dev, reqs[i].batch, reqs[i].output_dev, stream);
    out[i].status = st;
    if (st == TP_OK) {
      hipError_t e = hipEventRecord(c->trace_ev[i % kRing], stream);
      if (e != hipSuccess) {
        st = TP_E_HIP;
        out[i].status = st;
      }
    }
    if (st != TP_OK) {
      out[i].done_ns = out[i].issue_ns;
      if (first_err == TP_OK) {
        first_err = st;
        first_msg = last_error();
      }
      continue;
    }
    std::lock_guard<std::mutex> lk(mu);
    pending.push_back(i);
    ++in_flight;
    cv.notify_all();
  }
  {
    std::lock_guard<std::mutex> lk(mu);
    finished = true;
    cv.notify_all();
  }
  waiter.join();
  if (sync_err != hipSuccess) return fail(TP_E_HIP, std::string("tp_run_trace: ") + hipGetErrorString(sync_err));
  if (first_err != TP_OK) return fail(first_err, "tp_run_trace: a request failed: " + first_msg);
  return ok();
}
