// Implementation table: for each subkernel family, the implementations that
// can run a matched group, their launch counts and scratch needs.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "plan.hpp"

namespace mk {

bool impl_exists(const Plan& p, const Subkernel& sk, int impl);
int impl_launches(const Plan& p, const Subkernel& sk, int impl);
int64_t impl_scratch(const Plan& p, const Subkernel& sk, int impl);
// Largest scratch over the implementations of sk (so a swap never needs a
// bigger workspace).
int64_t max_scratch_bytes(const Plan& p, const Subkernel& sk);
// Whether the implementation runs its contraction on the matrix cores.
bool impl_uses_mfma(const Plan& p, const Subkernel& sk, int impl);
// mk_tuned_limit of the tuned implementation on this subkernel.
int tuned_limit(const Plan& p, const Subkernel& sk);

// Optional launch-level timing: brackets each kernel launch with a pair of
// HIP events taken from a pre-created pool (no synchronisation).
struct LaunchTimer {
  std::vector<hipEvent_t>* events = nullptr;  // 2 per recorded launch
  size_t next = 0;                            // next free event
  hipStream_t stream = nullptr;
  int only = -1;      // >= 0: record only this launch index of each run
  int pos = 0;        // launch index within the current run
  bool on = false;    // the current launch is being recorded
  void begin() {
    const int idx = pos++;
    on = events && next + 2 <= events->size() && (only < 0 || idx == only);
    if (on) (void)hipEventRecord((*events)[next++], stream);
  }
  void end() {
    if (on) (void)hipEventRecord((*events)[next++], stream);
    on = false;
  }
};

// Enqueue subkernel sk.  vals[v] is the device pointer of value v (null for
// values no buffer holds), out the subkernel's output buffer.
mk_status run_subkernel(const Plan& p, const Subkernel& sk, const std::vector<void*>& vals,
                        void* out, void* scratch, hipStream_t st, LaunchTimer* timer);

}  // namespace mk
