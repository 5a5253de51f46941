// Kernel timing probes shared by the host libraries: launches of selected
// kernel classes are bracketed with HIP events on the library's stream, and
// their algorithmic FLOPs and bytes are added up per class. Events are pooled
// so that a timed region creates none after the first pass.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

template <int NCLASS>
struct ProbeSet {
  struct Rec {
    hipEvent_t a, b;
    int cls;
  };
  uint32_t mask = 0;
  std::vector<Rec> live;
  std::vector<hipEvent_t> pool;
  double ms[NCLASS] = {}, flops[NCLASS] = {}, bytes[NCLASS] = {};
  int64_t launches[NCLASS] = {};

  hipEvent_t get_event() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }

  // Launch through f() on `stream`; bracket it with events when its class is enabled.
  template <class Fn>
  hipError_t run(hipStream_t stream, int cls, double fl, double by, Fn f) {
    const bool on = (mask >> cls) & 1u;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (on) {
      e0 = get_event();
      e1 = get_event();
      if (e0 && e1) (void)hipEventRecord(e0, stream);
    }
    hipError_t e = f();
    if (on && e0 && e1) {
      (void)hipEventRecord(e1, stream);
      live.push_back({e0, e1, cls});
      flops[cls] += fl;
      bytes[cls] += by;
      launches[cls] += 1;
    }
    return e;
  }

  // Fold the elapsed times of the recorded launches into the totals (waits for them).
  hipError_t collect() {
    for (auto& r : live) {
      hipError_t e = hipEventSynchronize(r.b);
      if (e != hipSuccess) return e;
      float t = 0.0f;
      e = hipEventElapsedTime(&t, r.a, r.b);
      if (e != hipSuccess) return e;
      ms[r.cls] += t;
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    live.clear();
    return hipSuccess;
  }

  hipError_t reset() {
    for (auto& r : live) {
      hipError_t e = hipEventSynchronize(r.b);
      if (e != hipSuccess) return e;
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    live.clear();
    for (int k = 0; k < NCLASS; ++k) {
      ms[k] = flops[k] = bytes[k] = 0.0;
      launches[k] = 0;
    }
    return hipSuccess;
  }

  ~ProbeSet() {
    for (auto& r : live) {
      (void)hipEventSynchronize(r.b);
      (void)hipEventDestroy(r.a);
      (void)hipEventDestroy(r.b);
    }
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
};
