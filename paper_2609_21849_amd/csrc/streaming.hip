// streaming.hip -- weight streaming: the executor that overlaps host-to-device
// copies of packed weights with the GEMMs, and the host-side model and
// planner of that schedule (paper Sec. 4, weight-streaming paragraph).
//
// Executor: a streamed layer's packed weight is copied into the next of a
// few device slots on a copy stream. Two events per slot order it: the copy
// waits for the slot's previous GEMM (slot_free) and the GEMM waits for the
// copy (slot_ready). The host only enqueues; both streams run ahead on their
// own, so the copy of a later layer proceeds under the GEMMs of earlier ones.
//
// Model: the same schedule as a discrete-event simulation (one copy engine,
// first come first served), used to predict step times and to plan which
// layers stay resident under a device memory budget (every subset for up to
// 16 layers; beyond that a greedy search under each slot-size cap).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "checks.hpp"
#include "kernels.hpp"
#include "log.hpp"
#include "qgemm.h"

namespace {

struct Sim {
  const double* w;
  const double* c;
  int n;
  int slots;
  double rate;
};

// Duration of the last of `steps` passes for the resident flags `res`.
double simulate(const Sim& s, const uint8_t* res, int steps) {
  std::vector<double> done;  // compute finish time of every streamed occurrence
  done.reserve((size_t)s.n * steps);
  double copy_idle = 0.0, t = 0.0, prev_end = 0.0, last = 0.0;
  for (int p = 0; p < steps; ++p) {
    for (int i = 0; i < s.n; ++i) {
      double ready = 0.0;
      if (!res[i]) {
        const size_t occ = done.size();
        const double slot_idle = occ >= (size_t)s.slots ? done[occ - s.slots] : 0.0;
        copy_idle = std::max(copy_idle, slot_idle) + s.w[i] / s.rate;
        ready = copy_idle;
      }
      t = std::max(t, ready) + s.c[i];
      if (!res[i]) done.push_back(t);
    }
    last = t - prev_end;
    prev_end = t;
  }
  return last;
}

double plan_bytes(const Sim& s, const uint8_t* res, double act) {
  double r = 0.0, wmax = 0.0;
  bool any = false;
  for (int i = 0; i < s.n; ++i) {
    if (res[i]) r += s.w[i];
    else { wmax = std::max(wmax, s.w[i]); any = true; }
  }
  return r + (any ? s.slots * wmax : 0.0) + act;
}

bool finite_nonneg(double v) { return v >= 0.0 && v <= 1e300; }

}  // namespace

extern "C" {

qg_status qg_stream_simulate(int32_t n_layers, const double* w_bytes, const double* compute_s,
                             const uint8_t* resident, int32_t n_slots, double h2d_bytes_per_s,
                             int32_t steps, double* step_s) {
  const qg_status st_ = [&]() -> qg_status {
    if (n_layers < 0 || steps < 1 || step_s == nullptr || !(h2d_bytes_per_s > 0.0)) return QG_ERR_INVALID_ARG;
    if (n_layers > 0 && (w_bytes == nullptr || compute_s == nullptr || resident == nullptr)) return QG_ERR_INVALID_ARG;
    bool streamed = false;
    for (int i = 0; i < n_layers; ++i) {
      if (!finite_nonneg(w_bytes[i]) || !finite_nonneg(compute_s[i])) return QG_ERR_INVALID_ARG;
      streamed |= !resident[i];
    }
    if (streamed && n_slots < 1) return QG_ERR_INVALID_ARG;
    const Sim s{w_bytes, compute_s, n_layers, n_slots, h2d_bytes_per_s};
    *step_s = simulate(s, resident, steps);
    return QG_OK;
  }();
  if (qg::log_enabled())
    qg::log_call("qg_stream_simulate", st_, "n_layers=%d n_slots=%d h2d=%.4g B/s steps=%d",
                 n_layers, n_slots, h2d_bytes_per_s, steps);
  return st_;
}

qg_status qg_stream_plan(int32_t n_layers, const double* w_bytes, const double* compute_s, int32_t n_slots,
                         double h2d_bytes_per_s, double budget_bytes, double act_peak_bytes,
                         uint8_t* resident_out, double* step_s, double* device_bytes) {
  const qg_status st_ = [&]() -> qg_status {
    if (n_layers < 0 || n_slots < 1 || !(h2d_bytes_per_s > 0.0) || !finite_nonneg(act_peak_bytes) ||
        !(budget_bytes >= 0.0) || step_s == nullptr || device_bytes == nullptr)
      return QG_ERR_INVALID_ARG;
    if (n_layers > 0 && (w_bytes == nullptr || compute_s == nullptr || resident_out == nullptr))
      return QG_ERR_INVALID_ARG;
    for (int i = 0; i < n_layers; ++i)
      if (!finite_nonneg(w_bytes[i]) || !finite_nonneg(compute_s[i])) return QG_ERR_INVALID_ARG;
    const Sim s{w_bytes, compute_s, n_layers, n_slots, h2d_bytes_per_s};
    constexpr int kPasses = 3;
    double compute_sum = 0.0;
    for (int i = 0; i < n_layers; ++i) compute_sum += compute_s[i];
    std::vector<uint8_t> res(n_layers, 0), best_res;
    double best_t = 0.0, best_b = 0.0;
    bool found = false;
    // a plan is better with a shorter step (relative 1e-12), then fewer bytes
    auto consider = [&](const std::vector<uint8_t>& r) {
      const double b = plan_bytes(s, r.data(), act_peak_bytes);
      if (b > budget_bytes) return;
      const double t = simulate(s, r.data(), kPasses);
      const double tol = 1e-12 * std::max(t, best_t);
      if (!found || t < best_t - tol || (t <= best_t + tol && b < best_b)) {
        found = true;
        best_t = t;
        best_b = b;
        best_res = r;
      }
    };
    if (n_layers <= 16) {
      // every resident subset
      for (uint32_t bits = 0; bits < (1u << n_layers); ++bits) {
        for (int i = 0; i < n_layers; ++i) res[i] = (bits >> i) & 1u;
        consider(res);
      }
    } else {
      // The streaming slots are as large as the largest streamed weight, so
      // fix that cap first: every layer above it is resident. Under each cap
      // (and with nothing streamed), add residents greedily by step time saved
      // per byte while they fit and copies are exposed.
      std::vector<double> caps(w_bytes, w_bytes + n_layers);
      std::sort(caps.begin(), caps.end());
      caps.erase(std::unique(caps.begin(), caps.end()), caps.end());
      std::fill(res.begin(), res.end(), 1);
      consider(res);
      for (double cap : caps) {
        for (int i = 0; i < n_layers; ++i) res[i] = w_bytes[i] > cap;
        if (plan_bytes(s, res.data(), act_peak_bytes) > budget_bytes) continue;
        double t = simulate(s, res.data(), kPasses), bytes = plan_bytes(s, res.data(), act_peak_bytes);
        consider(res);
        while (t > compute_sum * (1.0 + 1e-12)) {
          int pick = -1;
          double pick_gain = 0.0, pick_t = t, pick_b = bytes;
          for (int i = 0; i < n_layers; ++i) {
            if (res[i]) continue;
            res[i] = 1;
            const double b = plan_bytes(s, res.data(), act_peak_bytes);
            if (b <= budget_bytes) {
              const double ti = simulate(s, res.data(), kPasses);
              const double saved = t - ti, added = std::max(b - bytes, 1.0);
              if (saved > 0.0 && (pick < 0 || saved / added > pick_gain)) {
                pick = i;
                pick_gain = saved / added;
                pick_t = ti;
                pick_b = b;
              }
            }
            res[i] = 0;
          }
          if (pick < 0) break;
          res[pick] = 1;
          t = pick_t;
          bytes = pick_b;
          consider(res);
        }
      }
    }
    if (!found) return QG_ERR_BUFFER_TOO_SMALL;
    res = best_res;
    const double t = best_t, bytes = best_b;
    std::copy(res.begin(), res.end(), resident_out);
    *step_s = t;
    *device_bytes = bytes;
    return QG_OK;
  }();
  if (qg::log_enabled())
    qg::log_call("qg_stream_plan", st_, "n_layers=%d n_slots=%d h2d=%.4g B/s budget=%.4g B act=%.4g B",
                 n_layers, n_slots, h2d_bytes_per_s, budget_bytes, act_peak_bytes);
  return st_;
}

qg_status qg_run_layers(const qg_stream_layer* layers, int32_t n_layers, void* const* slots, int32_t n_slots,
                        size_t slot_bytes, void* const* slot_ready, void* const* slot_free, int32_t* slot_cursor,
                        void* compute_stream, void* copy_stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (n_layers < 0 || (n_layers > 0 && layers == nullptr)) return QG_ERR_INVALID_ARG;
    bool streamed = false;
    for (int i = 0; i < n_layers; ++i) streamed |= (layers[i].resident == 0);
    if (streamed) {
      if (n_slots < 1 || slots == nullptr || slot_ready == nullptr || slot_free == nullptr || slot_cursor == nullptr)
        return QG_ERR_INVALID_ARG;
      if (*slot_cursor < 0 || *slot_cursor >= n_slots) return QG_ERR_INVALID_ARG;
      for (int s = 0; s < n_slots; ++s)
        if (slots[s] == nullptr || (reinterpret_cast<uintptr_t>(slots[s]) & 255) != 0 || slot_ready[s] == nullptr ||
            slot_free[s] == nullptr)
          return QG_ERR_INVALID_ARG;
    }
    // every layer is checked before anything is enqueued; a streamed layer's
    // GEMM reads its weight from a slot, so the slot stands in for w_packed
    for (int i = 0; i < n_layers; ++i) {
      const qg_stream_layer& L = layers[i];
      if (L.a_fmt != QG_FMT_BF16) {
        const qg_status q = qg::check_quantize(L.a_fmt, L.x, L.m, L.k, L.k, L.a_codes, L.a_block_scales,
                                               L.a_tensor_scale);
        if (q != QG_OK) return q;
      }
      const void* wdev = L.resident ? L.w_packed : slots[0];
      if (!L.resident) {
        if (L.w_packed == nullptr) return QG_ERR_INVALID_ARG;
        if (L.w_packed_bytes > slot_bytes) return QG_ERR_BUFFER_TOO_SMALL;
      }
      const bool bf16 = (L.a_fmt == QG_FMT_BF16);
      if (L.y_dtype != QG_OUT_BF16 && L.y_dtype != QG_OUT_F32) return QG_ERR_INVALID_ARG;
      const qg_status g = qg::check_gemm(L.a_fmt, bf16 ? L.x : L.a_codes, bf16 ? nullptr : L.a_block_scales,
                                         bf16 ? nullptr : L.a_tensor_scale, L.k, L.w_fmt, wdev, L.w_packed_bytes,
                                         L.m, L.n, L.k, L.y, L.n, L.y_dtype == QG_OUT_F32 ? 4 : 2);
      if (g != QG_OK) return g;
    }
    hipStream_t cs = reinterpret_cast<hipStream_t>(compute_stream);
    hipStream_t xs = reinterpret_cast<hipStream_t>(copy_stream);
    int cur = streamed ? *slot_cursor : 0;
    for (int i = 0; i < n_layers; ++i) {
      const qg_stream_layer& L = layers[i];
      hipError_t e = hipSuccess;
      const bool bf16 = (L.a_fmt == QG_FMT_BF16);
      if (!bf16) {
        e = qg::launch_quantize((int)L.a_fmt, reinterpret_cast<const uint16_t*>(L.x), L.m, L.k, L.k,
                                reinterpret_cast<uint8_t*>(L.a_codes), reinterpret_cast<uint8_t*>(L.a_block_scales),
                                L.a_tensor_scale, cs);
        if (e != hipSuccess) return qg::status_of(e);
      }
      const void* wdev = L.w_packed;
      hipEvent_t ready = nullptr, free_ev = nullptr;
      if (!L.resident) {
        ready = reinterpret_cast<hipEvent_t>(slot_ready[cur]);
        free_ev = reinterpret_cast<hipEvent_t>(slot_free[cur]);
        wdev = slots[cur];
        if ((e = hipStreamWaitEvent(xs, free_ev, 0)) != hipSuccess) return qg::status_of(e);
        if ((e = hipMemcpyAsync(slots[cur], L.w_packed, L.w_packed_bytes, hipMemcpyHostToDevice, xs)) != hipSuccess)
          return qg::status_of(e);
        if ((e = hipEventRecord(ready, xs)) != hipSuccess) return qg::status_of(e);
        if ((e = hipStreamWaitEvent(cs, ready, 0)) != hipSuccess) return qg::status_of(e);
        cur = (cur + 1) % n_slots;
      }
      e = qg::launch_gemm((int)L.a_fmt, bf16 ? L.x : L.a_codes,
                          reinterpret_cast<const uint8_t*>(bf16 ? nullptr : L.a_block_scales),
                          bf16 ? nullptr : L.a_tensor_scale, L.k, reinterpret_cast<const uint8_t*>(wdev), L.m, L.n,
                          L.k, L.y, L.n, L.y_dtype == QG_OUT_F32 ? 1 : 0, nullptr, nullptr, cs);
      if (e != hipSuccess) return qg::status_of(e);
      if (!L.resident && (e = hipEventRecord(free_ev, cs)) != hipSuccess) return qg::status_of(e);
    }
    if (streamed) *slot_cursor = cur;
    return QG_OK;
  }();
  if (qg::log_enabled())
    qg::log_call("qg_run_layers", st_, "n_layers=%d n_slots=%d slot_bytes=%zu",
                 n_layers, n_slots, slot_bytes);
  return st_;
}

}  // extern "C"
