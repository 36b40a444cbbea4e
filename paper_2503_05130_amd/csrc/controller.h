// Quota controller: the paper's fast scale-up/down control (Sec. 3.4.1,
// Alg. 2) with CUs as tokens.  Pure host code.
//
// Every control period each co-located instance reports the kernels it
// launched during the period and the duration of its last iteration (the
// kernel launching cycle, KLC: one batch for an inference instance).  issue()
// then computes each instance's token issue R_issue from a transition table
// (controller.cpp): an SLO-sensitive instance's condition in the period
// (violation, idle, alone, sharing) sets the shared state and its own token
// rule, and the shared state sets the other instances' rule.  Only the
// instance that raised EMERGENCY can change the state again.  SLO-sensitive
// instances are evaluated first (they set the state), then the others, each
// group in id order.
//
// Tokens become quotas: round(R / granule) * granule clamped to
// [min_quota, MaxTokens], then fitted so that no two instances share a CU:
// SLO-sensitive quotas are scaled (granule, >= min_quota) until every other
// instance can keep min_quota, and the others are scaled into the CUs that
// remain.  SLO-sensitive instances take mask bits upward from 0 (id order),
// the others downward from the top (id order).
#pragma once

#include <cstdint>
#include <deque>
#include <vector>

namespace iefwd {

class QuotaController {
public:
    enum State : int32_t { None = 0, Emergency = 1, Recovery = 2, Contention = 3 };

    struct Params {
        uint32_t max_tokens = 256;   // MaxTokens: CUs (the device's CU count)
        uint32_t window = 4;         // RW length in control periods
        uint32_t granule = 8;        // quota granularity in CUs (one per XCD)
        uint32_t min_quota = 8;      // smallest quota issued
        double eta_violation = 0.2;  // relative KLC increase that raises EMERGENCY
        double eta_increase = 1.25;  // multiplicative scale-up per period
        bool temporary_yield = false;  // an EMERGENCY yield leaves R_last (the plan) unchanged
    };

    explicit QuotaController(const Params &p) : p_(p) {}

    // Adds an instance; returns its id (0, 1, ...).
    uint32_t add(double request, double limit, bool slo_sensitive);
    uint32_t size() const { return (uint32_t)insts_.size(); }

    // Observation for the current period: kernels launched during it and the
    // KLC of the last iteration completed in it (<= 0: none completed).
    void report(uint32_t id, uint64_t kernels, double klc_ms);

    // Ends the period: R_issue per instance (id order), then quotas and the
    // first mask bit of each placement.
    void issue(std::vector<double> &tokens, std::vector<uint32_t> &quotas, std::vector<uint32_t> &firsts);

    State state() const { return state_; }

private:
    struct Inst {
        double request, limit;
        bool slo;
        std::deque<uint64_t> rw;      // kernels per period, newest last
        uint64_t r_current = 0;
        double r_last = 0;
        double t_current = 0;   // KLC of this period; 0: none reported in it
        double t_min = -1;      // < 0: no KLC reported yet
        double dt = 0;
    };
    double issue_slo(uint32_t i);
    double issue_other(uint32_t i) const;
    double tokens_by_rule(int rule, const Inst &in) const;
    static uint64_t window_sum(const Inst &in);

    Params p_;
    std::vector<Inst> insts_;
    State state_ = None;
    int64_t owner_ = -1;   // instance that raised EMERGENCY
    double owner_dt_ = 0;
};

}  // namespace iefwd
