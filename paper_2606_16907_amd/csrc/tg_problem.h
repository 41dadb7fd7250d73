// tg_problem.h -- host-side definition of the opaque tg_problem handle.
#pragma once

#include <mutex>
#include <vector>

#include "tg_device.h"

struct tg_problem {
    int device;                  // device that was current at create
    tg::DevProblem P;            // device tables (one allocation, dev_block)
    void *dev_block;
    std::vector<int64_t> bvals;  // compatible micro-batch sizes, ascending
    int64_t n_compat_cfg;
    int64_t B;                    // global batch
    std::vector<int64_t> outact;  // [L] output activation bytes (host copy)
    std::vector<double> E;        // [K*K] inter-island bandwidth (host copy)
    // pinned host memory for the relaxed composition's packed read-backs and
    // uploads: allocated at its first call, grown when a call needs more,
    // freed at destroy; relaxed calls on one handle take turns on it
    mutable std::mutex relax_mu;
    mutable tg::HostStage relax_stage;
    mutable hipEvent_t relax_ev = nullptr;  // for the read-back of the fill depth limits
    // pinned words for the small read-backs of the prune (survivor count) and
    // the composition (fill depth limits, then the result), and an event for
    // the composition's overlapped one: taken by one call at a time (a call
    // that finds them busy reads back into pageable memory), freed at destroy
    mutable std::mutex readback_mu;
    mutable tg::HostStage readback_stage;
    mutable hipEvent_t compose_ev = nullptr;
};
