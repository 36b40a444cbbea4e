#include "quota.h"

#include <algorithm>

namespace iefwd {

bool build_cu_mask(uint32_t n_cu, uint32_t n_xcd, uint32_t q, uint32_t first, uint32_t *mask, uint32_t n_words) {
    if (!mask || n_cu == 0 || n_xcd == 0 || n_cu % n_xcd != 0 || q == 0 || q > n_cu || first >= n_cu ||
        n_words < mask_words(n_cu))
        return false;
    std::fill(mask, mask + n_words, 0u);
    // mask bit b is CU b / n_xcd of XCD b % n_xcd, so any run of consecutive
    // bits (cyclically) takes an equal share of every XCD, within one CU
    for (uint32_t i = 0; i < q; ++i) {
        const uint32_t bit = (first + i) % n_cu;
        mask[bit / 32] |= 1u << (bit % 32);
    }
    return true;
}

uint32_t mask_popcount(const std::vector<uint32_t> &mask, uint32_t n_cu) {
    uint32_t n = 0;
    for (uint32_t b = 0; b < n_cu && b / 32 < mask.size(); ++b) n += (mask[b / 32] >> (b % 32)) & 1u;
    return n;
}

MaskedStreams::~MaskedStreams() { clear(); }

void MaskedStreams::clear() {
    std::lock_guard<std::mutex> lock(mu_);
    for (Entry &e : entries_) {
        (void)hipStreamSynchronize(e.stream);
        (void)hipStreamDestroy(e.stream);
    }
    entries_.clear();
    current_ = nullptr;
}

hipStream_t MaskedStreams::find_locked(const std::vector<uint32_t> &mask) {
    ++clock_;
    for (Entry &e : entries_) {
        if (e.mask == mask) {
            e.last_use = clock_;
            return e.stream;
        }
    }
    return nullptr;
}

// Adds s for mask (or, if another thread added that mask meanwhile, destroys
// s and returns the cached one), evicting the least recently used stream that
// is not in use.
hipError_t MaskedStreams::insert_locked(const std::vector<uint32_t> &mask, hipStream_t s, hipStream_t *out) {
    if (hipStream_t have = find_locked(mask)) {
        (void)hipStreamDestroy(s);
        *out = have;
        return hipSuccess;
    }
    if (entries_.size() >= capacity_) {
        size_t victim = entries_.size();
        for (size_t i = 0; i < entries_.size(); ++i) {
            if (entries_[i].stream == current_) continue;
            if (victim == entries_.size() || entries_[i].last_use < entries_[victim].last_use) victim = i;
        }
        if (victim < entries_.size()) {
            hipError_t err = hipStreamSynchronize(entries_[victim].stream);
            if (err != hipSuccess) return err;
            err = hipStreamDestroy(entries_[victim].stream);
            if (err != hipSuccess) return err;
            entries_.erase(entries_.begin() + (long)victim);
        }
    }
    entries_.push_back(Entry{mask, s, clock_});
    *out = s;
    return hipSuccess;
}

hipError_t MaskedStreams::get(const std::vector<uint32_t> &mask, hipStream_t *out) {
    {
        std::lock_guard<std::mutex> lock(mu_);
        if ((*out = find_locked(mask))) return hipSuccess;
    }
    hipStream_t s = nullptr;   // created without holding the lock
    hipError_t err = hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data());
    if (err != hipSuccess) return err;
    std::lock_guard<std::mutex> lock(mu_);
    return insert_locked(mask, s, out);
}

hipError_t MaskedStreams::acquire(const std::vector<uint32_t> &mask, hipStream_t *out) {
    hipError_t err = get(mask, out);
    if (err != hipSuccess) return err;
    std::lock_guard<std::mutex> lock(mu_);
    // re-check: a concurrent prepare() may have evicted it between get() and here
    if (hipStream_t have = find_locked(mask)) {
        *out = have;
    } else {
        hipStream_t s = nullptr;
        err = hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data());
        if (err != hipSuccess) return err;
        err = insert_locked(mask, s, out);
        if (err != hipSuccess) return err;
    }
    current_ = *out;
    return hipSuccess;
}

hipError_t MaskedStreams::set_capacity(size_t capacity) {
    std::lock_guard<std::mutex> lock(mu_);
    capacity_ = capacity < 1 ? 1 : capacity;
    while (entries_.size() > capacity_) {
        size_t victim = entries_.size();
        for (size_t i = 0; i < entries_.size(); ++i) {
            if (entries_[i].stream == current_) continue;
            if (victim == entries_.size() || entries_[i].last_use < entries_[victim].last_use) victim = i;
        }
        if (victim == entries_.size()) break;
        hipError_t err = hipStreamSynchronize(entries_[victim].stream);
        if (err != hipSuccess) return err;
        err = hipStreamDestroy(entries_[victim].stream);
        if (err != hipSuccess) return err;
        entries_.erase(entries_.begin() + (long)victim);
    }
    return hipSuccess;
}

hipError_t MaskedStreams::prepare(const std::vector<uint32_t> &mask) {
    hipStream_t s = nullptr;
    return get(mask, &s);
}

}  // namespace iefwd
