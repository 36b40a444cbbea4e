// Compute quota as a CU mask on the instance's HIP stream.
//
// The paper scales each co-located instance's compute share up and down at
// run time in continuous (non-integer) fractions of a GPU (Sec. 3.4), with a
// share changing between iterations (Alg. 2 issues a new share every control
// period).  Here a share of q CUs is a hardware queue whose CU mask enables q
// CUs spread evenly over the XCDs; a change of quota switches the instance to
// another (cached) masked stream at the next batch boundary.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

namespace iefwd {

// Mask words for q CUs out of n_cu in n_xcd XCDs: mask bits first, first + 1,
// ..., first + q - 1 (mod n_cu).  Mask bit b drives the CU with index
// b / n_xcd inside XCD b % n_xcd (the driver hands mask bits to the XCDs
// round-robin), so every XCD gets q / n_xcd CUs or one more; with first = 0,
// XCD x gets the extra CU if x < q % n_xcd.  Instances placed at first = 0,
// q0, q0 + q1, ... get disjoint CUs while the quotas sum to at most n_cu.
// Returns false if the arguments are out of range.
bool build_cu_mask(uint32_t n_cu, uint32_t n_xcd, uint32_t q, uint32_t first, uint32_t *mask, uint32_t n_words);

inline uint32_t mask_words(uint32_t n_cu) { return (n_cu + 31) / 32; }

uint32_t mask_popcount(const std::vector<uint32_t> &mask, uint32_t n_cu);

// Small LRU cache of CU-masked streams for one instance.  Creating a masked
// stream creates a hardware queue (about 5 ms on MI355X), so it is kept off
// the batch path: once a mask has been seen, or prepared ahead of time from
// another thread, switching to it costs one event wait.  Measured on MI355X:
// creating or destroying a masked queue stalls the work of every other queue
// of the process for about 3 ms (the hardware scheduler rewrites its queue
// list), and with more than about 20-24 live queues in a process the
// scheduler time-slices them (batches stall 12-33 ms).  So the cache is
// small (2 by default: the stream in use and the next one) and a serving
// loop should switch among a fixed set of prepared masks.  Streams are
// created at the default priority.  Thread-safe: prepare() may run
// concurrently with acquire(); stream creation happens outside the lock.
class MaskedStreams {
public:
    explicit MaskedStreams(size_t capacity = 2) : capacity_(capacity) {}
    MaskedStreams(const MaskedStreams &) = delete;
    MaskedStreams &operator=(const MaskedStreams &) = delete;
    ~MaskedStreams();

    // The stream with exactly this mask (created if missing); it becomes the
    // stream in use, which is never evicted until another one is acquired.
    hipError_t acquire(const std::vector<uint32_t> &mask, hipStream_t *out);
    // Makes sure a stream with this mask is cached (creating it if missing)
    // without changing the stream in use.
    hipError_t prepare(const std::vector<uint32_t> &mask);
    // Keeps at most `capacity` streams (>= 1), destroying the least recently
    // used ones beyond it (never the stream in use).
    hipError_t set_capacity(size_t capacity);
    void clear();   // synchronises and destroys every cached stream

private:
    struct Entry {
        std::vector<uint32_t> mask;
        hipStream_t stream;
        uint64_t last_use;
    };
    hipStream_t find_locked(const std::vector<uint32_t> &mask);
    hipError_t insert_locked(const std::vector<uint32_t> &mask, hipStream_t s, hipStream_t *out);
    hipError_t get(const std::vector<uint32_t> &mask, hipStream_t *out);

    std::mutex mu_;
    std::vector<Entry> entries_;
    size_t capacity_;
    uint64_t clock_ = 0;
    hipStream_t current_ = nullptr;
};

}  // namespace iefwd
