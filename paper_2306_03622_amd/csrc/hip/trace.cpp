// Open-loop trace replay (tp_run_trace): the calling thread issues requests at their
// arrival times; a completion thread waits for each request's event in issue order.
#include <hip/hip_runtime_api.h>

#include <chrono>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>

#include <map>

#include "../core/errors.hpp"
#include "../core/sched.hpp"
#include "runtime.hpp"

using namespace tp;

namespace {

constexpr uint32_t kRing = 256;

uint64_t since(std::chrono::steady_clock::time_point t0) {
  return (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - t0)
      .count();
}

// Waits until `when`: sleeps until shortly before it, then spins, so that a request is issued
// within a few microseconds of its arrival instead of after the sleep's wake-up delay (timer
// slack and scheduling, tens of microseconds), which would count as latency.
constexpr auto kSpin = std::chrono::microseconds(200);
void wait_until(std::chrono::steady_clock::time_point when) {
  if (std::chrono::steady_clock::now() + kSpin < when) std::this_thread::sleep_until(when - kSpin);
  while (std::chrono::steady_clock::now() < when) {
  }
}

tp_status make_ring(tp_ctx* c) {
  if (!c->trace_ev.empty()) return TP_OK;
  c->trace_ev.assign(kRing, nullptr);
  for (auto& e : c->trace_ev) {
    hipError_t err = hipEventCreateWithFlags(&e, hipEventDisableTiming);
    if (err != hipSuccess) {
      for (auto& x : c->trace_ev)
        if (x) (void)hipEventDestroy(x);
      c->trace_ev.clear();
      return fail(TP_E_HIP, std::string("trace replay: event creation: ") + hipGetErrorString(err));
    }
  }
  return TP_OK;
}

}  // namespace

extern "C" tp_status tp_run_trace(tp_ctx* c, const tp_request* reqs, uint32_t n, void* stream_,
                                  tp_request_result* out) {
  if (!c || (n && (!reqs || !out))) return fail(TP_E_INVAL, "tp_run_trace: NULL argument");
  for (uint32_t i = 1; i < n; ++i)
    if (reqs[i].arrival_ns < reqs[i - 1].arrival_ns) return fail(TP_E_INVAL, "tp_run_trace: arrivals must not decrease");
  if (make_ring(c) != TP_OK) return TP_E_HIP;
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
    wait_until(t0 + std::chrono::nanoseconds(reqs[i].arrival_ns));
    {
      std::unique_lock<std::mutex> lk(mu);
      cv.wait(lk, [&] { return in_flight < kRing; });
    }
    int32_t res = 0;
    (void)tp_is_resident(c, reqs[i].model_id, &res);
    out[i].hit = res;
    out[i].issue_ns = since(t0);
    const uint64_t calls = c->admit_calls;
    tp_status st = tp_infer(c, reqs[i].model_id, reqs[i].input_dev, reqs[i].batch, reqs[i].output_dev, stream);
    out[i].admit_ns = c->admit_calls != calls ? c->last_admit_ns : 0;
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

extern "C" tp_status tp_run_trace_sched(tp_ctx* c, const tp_request* reqs, uint32_t n, void* stream_,
                                        const tp_sched_config* cfg, const uint64_t* deadline_ns,
                                        tp_request_result* out, tp_sched_stats* stats) {
  if (!c || !cfg || (n && (!reqs || !out || !deadline_ns))) return fail(TP_E_INVAL, "tp_run_trace_sched: NULL argument");
  if ((cfg->policy != TP_QUEUE_FIFO && cfg->policy != TP_QUEUE_SLO) || cfg->max_inflight < 1 ||
      cfg->max_inflight > (int32_t)kRing || !(cfg->slo_pct > 0 && cfg->slo_pct < 1) ||
      !(cfg->alpha > 0 && cfg->alpha <= 1) || !(cfg->scalar > 1) || cfg->period_ns == 0)
    return fail(TP_E_INVAL, "tp_run_trace_sched: bad configuration");
  for (uint32_t i = 1; i < n; ++i)
    if (reqs[i].arrival_ns < reqs[i - 1].arrival_ns)
      return fail(TP_E_INVAL, "tp_run_trace_sched: arrivals must not decrease");
  if (make_ring(c) != TP_OK) return TP_E_HIP;
  // functions: the model ids of the trace, densely numbered in increasing id order
  std::map<int32_t, int32_t> fid;
  for (uint32_t i = 0; i < n; ++i) fid.emplace(reqs[i].model_id, 0);
  int32_t nf = 0;
  for (auto& kv : fid) kv.second = nf++;
  std::vector<int32_t> func(n);
  for (uint32_t i = 0; i < n; ++i) func[i] = fid[reqs[i].model_id];

  hipStream_t stream = static_cast<hipStream_t>(stream_);
  std::mutex mu;
  std::condition_variable cv;
  // enqueued on the GPU, awaiting completion, in issue order: (request, event slot); slots go
  // round the ring in issue order, and at most max_inflight <= kRing requests are in flight
  std::deque<std::pair<uint32_t, uint32_t>> issued;
  uint32_t issue_seq = 0;
  uint32_t in_flight = 0;
  bool finished = false;
  hipError_t sync_err = hipSuccess;
  // per function: served and within deadline, over the trace and in the current period
  std::vector<uint64_t> n_all(nf, 0), m_all(nf, 0), n_per(nf, 0), m_per(nf, 0);
  double alpha = cfg->alpha, last_ratio = -1.0;
  uint32_t periods = 0, changes = 0;
  uint64_t period_end = cfg->period_ns;
  const double p = cfg->slo_pct;
  const auto t0 = std::chrono::steady_clock::now();

  auto close_periods = [&](uint64_t now) {       // under mu
    while (now >= period_end) {
      uint32_t active = 0, good = 0;
      for (int32_t f = 0; f < nf; ++f) {
        if (!n_per[f]) continue;
        ++active;
        if ((double)m_per[f] >= p * (double)n_per[f]) ++good;
        n_per[f] = m_per[f] = 0;
      }
      if (active) {
        const double ratio = (double)good / active;
        if (last_ratio >= 0) {
          const double a = alpha_update(alpha, last_ratio, ratio, cfg->scalar, cfg->threshold);
          if (a != alpha) ++changes;
          alpha = a;
        }
        last_ratio = ratio;
      }
      ++periods;
      period_end += cfg->period_ns;
    }
  };

  std::thread waiter([&] {
    for (;;) {
      uint32_t i, slot;
      {
        std::unique_lock<std::mutex> lk(mu);
        cv.wait(lk, [&] { return !issued.empty() || finished; });
        if (issued.empty()) return;
        i = issued.front().first;
        slot = issued.front().second;
        issued.pop_front();
      }
      hipError_t e = hipEventSynchronize(c->trace_ev[slot]);
      const uint64_t t = since(t0);
      std::lock_guard<std::mutex> lk(mu);
      out[i].done_ns = t;
      if (e != hipSuccess && sync_err == hipSuccess) sync_err = e;
      close_periods(t);
      const int32_t f = func[i];
      const bool met = t - reqs[i].arrival_ns <= deadline_ns[i];
      ++n_all[f]; ++n_per[f];
      if (met) { ++m_all[f]; ++m_per[f]; }
      --in_flight;
      cv.notify_all();
    }
  });

  tp_status first_err = TP_OK;
  std::string first_msg;
  std::vector<uint32_t> queue;                  // arrived, not yet issued, in arrival order
  uint32_t next = 0;
  while (next < n || !queue.empty()) {
    {
      std::unique_lock<std::mutex> lk(mu);
      cv.wait(lk, [&] { return in_flight < (uint32_t)cfg->max_inflight; });
    }
    const uint64_t now = since(t0);
    while (next < n && reqs[next].arrival_ns <= now) queue.push_back(next++);
    if (queue.empty()) {
      wait_until(t0 + std::chrono::nanoseconds(reqs[next].arrival_ns));
      continue;
    }
    size_t k = 0;                               // FIFO: the earliest arrival
    if (cfg->policy == TP_QUEUE_SLO) {
      std::vector<double> r(nf);
      {
        std::lock_guard<std::mutex> lk(mu);
        close_periods(now);
        for (int32_t f = 0; f < nf; ++f) r[f] = rrc(n_all[f], m_all[f], p);
      }
      const std::vector<uint8_t> high = high_group(r, alpha);
      std::vector<int32_t> pend(queue.size());
      for (size_t q = 0; q < queue.size(); ++q) pend[q] = func[queue[q]];
      k = (size_t)sched_pick(r, high, pend);
    }
    const uint32_t i = queue[k];
    queue.erase(queue.begin() + k);
    int32_t res = 0;
    (void)tp_is_resident(c, reqs[i].model_id, &res);
    out[i].hit = res;
    out[i].issue_ns = since(t0);
    const uint32_t slot = issue_seq % kRing;
    const uint64_t calls = c->admit_calls;
    tp_status st = tp_infer(c, reqs[i].model_id, reqs[i].input_dev, reqs[i].batch, reqs[i].output_dev, stream);
    out[i].admit_ns = c->admit_calls != calls ? c->last_admit_ns : 0;
    if (st == TP_OK && hipEventRecord(c->trace_ev[slot], stream) != hipSuccess) st = TP_E_HIP;
    out[i].status = st;
    if (st != TP_OK) {
      out[i].done_ns = out[i].issue_ns;
      if (first_err == TP_OK) {
        first_err = st;
        first_msg = last_error();
      }
      continue;
    }
    std::lock_guard<std::mutex> lk(mu);
    issued.push_back({i, slot});
    ++issue_seq;
    ++in_flight;
    cv.notify_all();
  }
  {
    std::lock_guard<std::mutex> lk(mu);
    finished = true;
    cv.notify_all();
  }
  waiter.join();
  if (stats) {
    stats->alpha = alpha;
    stats->periods = periods;
    stats->alpha_changes = changes;
    stats->compliant = stats->functions = 0;
    for (int32_t f = 0; f < nf; ++f) {
      if (!n_all[f]) continue;
      ++stats->functions;
      if ((double)m_all[f] >= p * (double)n_all[f]) ++stats->compliant;
    }
  }
  if (sync_err != hipSuccess) return fail(TP_E_HIP, std::string("tp_run_trace_sched: ") + hipGetErrorString(sync_err));
  if (first_err != TP_OK) return fail(first_err, "tp_run_trace_sched: a request failed: " + first_msg);
  return ok();
}
