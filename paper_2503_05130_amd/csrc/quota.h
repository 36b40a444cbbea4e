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
// stream creates a hardware queue, so it is kept off the batch path once a
// mask has been seen.  Streams are created at the default priority.
class MaskedStreams {
public:
    explicit MaskedStreams(size_t capacity = 4) : capacity_(capacity) {}
    MaskedStreams(const MaskedStreams &) = delete;
    MaskedStreams &operator=(const MaskedStreams &) = delete;
    ~MaskedStreams();

    // Stream with exactly this mask (created on first use).  `keep` is never
    // evicted (the stream currently in use).
    hipError_t get(const std::vector<uint32_t> &mask, hipStream_t keep, hipStream_t *out);
    void clear();   // synchronises and destroys every cached stream

private:
    struct Entry {
        std::vector<uint32_t> mask;
        hipStream_t stream;
        uint64_t last_use;
    };
    std::vector<Entry> entries_;
    size_t capacity_;
    uint64_t clock_ = 0;
};

}  // namespace iefwd
