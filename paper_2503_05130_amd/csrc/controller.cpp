// Quota controller (Sec. 3.4.1, Alg. 2) on CU quotas; see controller.h.
#include "controller.h"

#include <algorithm>
#include <cmath>

namespace iefwd {

uint32_t QuotaController::add(double request, double limit, bool slo_sensitive) {
    Inst in{};
    in.request = request;
    in.limit = limit;
    in.slo = slo_sensitive;
    in.r_last = p_.max_tokens * request;
    insts_.push_back(in);
    return (uint32_t)insts_.size() - 1;
}

void QuotaController::report(uint32_t id, uint64_t kernels, double klc_ms) {
    Inst &in = insts_.at(id);
    in.r_current = kernels;
    if (klc_ms > 0) {
        in.t_current = klc_ms;
        in.t_min = in.t_min < 0 ? klc_ms : std::min(in.t_min, klc_ms);
    }
}

uint64_t QuotaController::window_sum(const Inst &in) {
    uint64_t s = 0;
    for (uint64_t v : in.rw) s += v;
    return s;
}

// Sec. 3.4.1 as a transition table.  Each period an SLO-sensitive instance's
// observations fall into one condition, checked in this order:
//   Violation  its KLC rose by more than eta_violation over its best (dT);
//   Idle       it launched no kernels in its window;
//   Alone      every co-located instance launched none in theirs;
//   Sharing    otherwise.
// The condition decides the shared state and the instance's own token rule;
// the shared state decides the other instances' rule.  Token rules:
//   LimitShare    MaxTokens * limit
//   RequestShare  MaxTokens * request
//   GrowToMax     R_last * eta_increase, at most MaxTokens
//   GrowToLimit   R_last * eta_increase, at most MaxTokens * limit
//   Yield         min(MaxTokens * request, R_last) / (1 + dT of the raiser)
//   Keep          R_last
// Readings where the paper's text leaves it open: Yield divides by the KLC
// ratio 1 + dT (a division by dT alone would scale up for dT < 1), GrowToMax is
// capped at MaxTokens, T_min is the smallest KLC over the whole history, and a
// period in which an instance completed no iteration has no T_current and dT 0
// (carrying the last KLC over would hold an instance that went idle after a
// violation in Violation, and the Idle condition could never follow it).
namespace {

enum class Condition { Violation, Idle, Alone, Sharing };
enum class Rule { LimitShare, RequestShare, GrowToMax, GrowToLimit, Yield, Keep };

struct Transition {
    QuotaController::State state;
    Rule rule;
};

// SLO-sensitive instance: condition -> (shared state, own rule)
constexpr Transition kSloTransition[] = {
    /* Violation */ {QuotaController::Emergency, Rule::LimitShare},
    /* Idle      */ {QuotaController::Recovery, Rule::RequestShare},
    /* Alone     */ {QuotaController::Recovery, Rule::GrowToMax},
    /* Sharing   */ {QuotaController::Contention, Rule::RequestShare},
};

// other instances: shared state -> rule
constexpr Rule kOtherRule[] = {
    /* None       */ Rule::LimitShare,
    /* Emergency  */ Rule::Yield,
    /* Recovery   */ Rule::GrowToLimit,
    /* Contention */ Rule::Keep,
};

}  // namespace

double QuotaController::tokens_by_rule(int rule, const Inst &in) const {
    const double maxt = p_.max_tokens;
    switch (static_cast<Rule>(rule)) {
    case Rule::LimitShare: return maxt * in.limit;
    case Rule::RequestShare: return maxt * in.request;
    case Rule::GrowToMax: return std::min(in.r_last * p_.eta_increase, maxt);
    case Rule::GrowToLimit: return std::min(in.r_last * p_.eta_increase, maxt * in.limit);
    case Rule::Yield: return std::min(maxt * in.request, in.r_last) / (1.0 + owner_dt_);
    case Rule::Keep: break;
    }
    return in.r_last;
}

double QuotaController::issue_slo(uint32_t i) {
    Inst &in = insts_[i];
    in.dt = in.t_current > 0 ? (in.t_current - in.t_min) / in.t_min : 0.0;
    bool others_idle = true;
    for (uint32_t j = 0; j < insts_.size(); ++j)
        if (j != i && window_sum(insts_[j]) != 0) others_idle = false;
    const Condition c = in.dt > p_.eta_violation ? Condition::Violation
                        : window_sum(in) == 0    ? Condition::Idle
                        : others_idle            ? Condition::Alone
                                                 : Condition::Sharing;
    const Transition t = kSloTransition[static_cast<int>(c)];
    // only the instance that raised EMERGENCY may move the state out of it
    if (state_ != Emergency || owner_ == (int64_t)i) {
        state_ = t.state;
        owner_ = t.state == Emergency ? (int64_t)i : -1;
        owner_dt_ = t.state == Emergency ? in.dt : 0.0;
    }
    return tokens_by_rule(static_cast<int>(t.rule), in);
}

double QuotaController::issue_other(uint32_t i) const {
    return tokens_by_rule(static_cast<int>(kOtherRule[state_]), insts_[i]);
}

void QuotaController::issue(std::vector<double> &tokens, std::vector<uint32_t> &quotas,
                            std::vector<uint32_t> &firsts) {
    const uint32_t n = (uint32_t)insts_.size();
    bool any_slo = false;
    for (Inst &in : insts_) {
        in.rw.push_back(in.r_current);
        while (in.rw.size() > p_.window) in.rw.pop_front();
        any_slo = any_slo || in.slo;
    }
    if (!any_slo) {
        state_ = None;
        owner_ = -1;
        owner_dt_ = 0;
    }
    tokens.assign(n, 0.0);
    for (uint32_t i = 0; i < n; ++i)
        if (insts_[i].slo) tokens[i] = issue_slo(i);
    for (uint32_t i = 0; i < n; ++i)
        if (!insts_[i].slo) tokens[i] = issue_other(i);
    // tokens -> quotas that never share a CU: SLO-sensitive quotas are scaled
    // so that every other instance keeps min_quota, the others are scaled into
    // what remains; SLO-sensitive instances are placed upward from mask bit 0,
    // the others downward from the top
    quotas.assign(n, 0);
    firsts.assign(n, 0);
    // the text calls the co-located instances' EMERGENCY scale-down temporary:
    // with temporary_yield their plan R_last survives it, so the yield does
    // not compound over consecutive EMERGENCY periods and CONTENTION restores
    // the plan; without it the yielded issue becomes R_last as in Alg. 2
    const bool yielded = state_ == Emergency && p_.temporary_yield;
    for (uint32_t i = 0; i < n; ++i) {
        if (insts_[i].slo || !yielded) insts_[i].r_last = tokens[i];
        insts_[i].r_current = 0;
        insts_[i].t_current = 0;   // a period with no completed iteration has no KLC
        const double units = std::floor(tokens[i] / p_.granule + 0.5);
        quotas[i] = (uint32_t)std::max<double>(p_.min_quota, std::min<double>(p_.max_tokens, units * p_.granule));
    }
    // shrink one group to at most `avail` CUs: min_quota each, the rest shared in
    // proportion to each quota's excess over min_quota (down to the granule)
    auto fit = [&](bool slo, int64_t avail) {
        uint64_t want = 0, count = 0;
        for (uint32_t i = 0; i < n; ++i)
            if (insts_[i].slo == slo) {
                want += quotas[i];
                ++count;
            }
        if (count == 0 || (int64_t)want <= avail) return;
        const int64_t spare_s = avail - (int64_t)(count * p_.min_quota);
        const uint64_t spare = spare_s > 0 ? (uint64_t)spare_s : 0;
        const uint64_t excess = want - count * p_.min_quota;
        for (uint32_t i = 0; i < n; ++i)
            if (insts_[i].slo == slo) {
                const uint64_t extra =
                    excess ? ((quotas[i] - p_.min_quota) * spare / excess) / p_.granule * p_.granule : 0;
                quotas[i] = p_.min_quota + (uint32_t)extra;
            }
    };
    int64_t n_other = 0, slo_sum = 0;
    for (uint32_t i = 0; i < n; ++i) n_other += insts_[i].slo ? 0 : 1;
    fit(true, (int64_t)p_.max_tokens - n_other * (int64_t)p_.min_quota);
    for (uint32_t i = 0; i < n; ++i) slo_sum += insts_[i].slo ? quotas[i] : 0;
    fit(false, (int64_t)p_.max_tokens - slo_sum);
    int64_t lo = 0, hi = p_.max_tokens;
    for (uint32_t i = 0; i < n; ++i) {
        if (insts_[i].slo) {
            firsts[i] = (uint32_t)(lo % p_.max_tokens);
            lo += quotas[i];
        }
    }
    for (uint32_t i = 0; i < n; ++i) {
        if (!insts_[i].slo) {
            hi -= quotas[i];
            firsts[i] = (uint32_t)(((hi % (int64_t)p_.max_tokens) + p_.max_tokens) % p_.max_tokens);
        }
    }
}

}  // namespace iefwd
