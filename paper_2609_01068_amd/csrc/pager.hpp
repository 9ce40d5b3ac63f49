// Host-side allocator of the paged draft KV cache and per-slot bookkeeping.
//
// Rule (the paper leaves allocation open; this one makes page tables unique):
// the free page with the lowest id is taken first; a prefill takes
// ceil(n / page_size) pages per request, requests in argument order; a decode
// step takes one page for a request exactly when its cached length is a
// multiple of page_size before the append; release returns the pages.
// Every check runs before any change, so a failed call changes nothing.
#pragma once

#include <cstdint>
#include <functional>
#include <queue>
#include <vector>

namespace outlets {

class Pager {
public:
    Pager(int32_t num_pages, int32_t page_size, int32_t max_slots, int32_t max_seq_len);

    // Status codes are the OUTLETS_* values of outlets.h.  On success,
    // `updates` (optional) receives (table index, page id) for every new
    // page-table entry, in allocation order.
    int prefill(int32_t n, const int32_t* slots, const int32_t* lens,
                std::vector<int32_t>* updates, const char** why);
    int step(int32_t n, const int32_t* slots, std::vector<int32_t>* updates,
             const char** why);
    // The checks of step() alone (same order and codes); changes nothing.
    int check_step(int32_t n, const int32_t* slots, const char** why);
    int release(int32_t n, const int32_t* slots, const char** why);

    int32_t max_pages_per_seq() const { return max_pages_; }
    int32_t max_slots() const { return max_slots_; }
    int32_t seq_len(int32_t s) const { return seq_len_[s]; }
    bool active(int32_t s) const { return seq_len_[s] > 0; }
    int32_t n_free() const { return static_cast<int32_t>(free_.size()); }
    const std::vector<int32_t>& table() const { return table_; }
    const std::vector<int32_t>& seq_lens() const { return seq_len_; }

private:
    int check_slots(int32_t n, const int32_t* slots, const char** why);
    int32_t take_lowest();

    int32_t page_size_, max_slots_, max_seq_len_, max_pages_;
    std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> free_;
    std::vector<int32_t> table_;    // [max_slots * max_pages], -1 = unused
    std::vector<int32_t> seq_len_;  // cached tokens per slot, 0 = inactive
    std::vector<uint8_t> mark_;     // scratch for repeated-slot detection
};

// Varlen offsets, positions and last-token rows of packed prompts.
int varlen_meta(int32_t n, const int32_t* lens, int32_t* cu, int32_t* pos, int32_t* last);

}  // namespace outlets
