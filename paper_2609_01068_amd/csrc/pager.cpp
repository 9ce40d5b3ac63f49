#include "pager.hpp"

#include "outlets.h"

namespace outlets {

Pager::Pager(int32_t num_pages, int32_t page_size, int32_t max_slots, int32_t max_seq_len)
    : page_size_(page_size), max_slots_(max_slots),
      max_seq_len_(max_seq_len), max_pages_((max_seq_len + page_size - 1) / page_size),
      table_(static_cast<size_t>(max_slots) * max_pages_, -1),
      seq_len_(max_slots, 0), mark_(max_slots, 0) {
    std::vector<int32_t> ids(num_pages);
    for (int32_t i = 0; i < num_pages; ++i) ids[i] = i;
    free_ = decltype(free_)(std::greater<int32_t>(), std::move(ids));
}

int32_t Pager::take_lowest() {
    int32_t p = free_.top();
    free_.pop();
    return p;
}

int Pager::check_slots(int32_t n, const int32_t* slots, const char** why) {
    int rc = OUTLETS_OK;
    int32_t i = 0;
    for (; i < n; ++i) {
        int32_t s = slots[i];
        if (s < 0 || s >= max_slots_) { *why = "slot out of range"; rc = OUTLETS_ERR_INVALID_ARG; break; }
        if (mark_[s]) { *why = "slot repeated in one call"; rc = OUTLETS_ERR_INVALID_ARG; break; }
        mark_[s] = 1;
    }
    for (int32_t j = 0; j < i; ++j) mark_[slots[j]] = 0;
    return rc;
}

int Pager::prefill(int32_t n, const int32_t* slots, const int32_t* lens,
                   std::vector<int32_t>* updates, const char** why) {
    // per request: slot range / repetition, then the length
    int rc = OUTLETS_OK;
    int32_t i = 0;
    for (; i < n; ++i) {
        int32_t s = slots[i];
        if (s < 0 || s >= max_slots_) { *why = "slot out of range"; rc = OUTLETS_ERR_INVALID_ARG; break; }
        if (mark_[s]) { *why = "slot repeated in one call"; rc = OUTLETS_ERR_INVALID_ARG; break; }
        mark_[s] = 1;
        if (lens[i] <= 0 || lens[i] > max_seq_len_) {
            *why = "prompt length must be in [1, max_seq_len]";
            rc = OUTLETS_ERR_INVALID_ARG;
            ++i;
            break;
        }
    }
    for (int32_t j = 0; j < i; ++j) mark_[slots[j]] = 0;
    if (rc != OUTLETS_OK) return rc;
    for (i = 0; i < n; ++i)
        if (active(slots[i])) { *why = "prefill on an active slot"; return OUTLETS_ERR_SLOT_BUSY; }
    int64_t need = 0;
    for (i = 0; i < n; ++i) need += (lens[i] + page_size_ - 1) / page_size_;
    if (need > n_free()) { *why = "KV page pool exhausted"; return OUTLETS_ERR_OUT_OF_PAGES; }
    for (i = 0; i < n; ++i) {
        int32_t s = slots[i];
        int32_t np = (lens[i] + page_size_ - 1) / page_size_;
        for (int32_t j = 0; j < np; ++j) {
            int32_t p = take_lowest();
            size_t idx = static_cast<size_t>(s) * max_pages_ + j;
            table_[idx] = p;
            if (updates) { updates->push_back(static_cast<int32_t>(idx)); updates->push_back(p); }
        }
        seq_len_[s] = lens[i];
    }
    return OUTLETS_OK;
}

int Pager::check_step(int32_t n, const int32_t* slots, const char** why) {
    int rc = check_slots(n, slots, why);
    if (rc != OUTLETS_OK) return rc;
    for (int32_t i = 0; i < n; ++i)
        if (!active(slots[i])) { *why = "step on an inactive slot"; return OUTLETS_ERR_SLOT_EMPTY; }
    for (int32_t i = 0; i < n; ++i)
        if (seq_len_[slots[i]] >= max_seq_len_) { *why = "slot is at max_seq_len"; return OUTLETS_ERR_INVALID_ARG; }
    int32_t need = 0;
    for (int32_t i = 0; i < n; ++i) need += (seq_len_[slots[i]] % page_size_ == 0);
    if (need > n_free()) { *why = "KV page pool exhausted"; return OUTLETS_ERR_OUT_OF_PAGES; }
    return OUTLETS_OK;
}

int Pager::step(int32_t n, const int32_t* slots, std::vector<int32_t>* updates, const char** why) {
    int rc = check_step(n, slots, why);
    if (rc != OUTLETS_OK) return rc;
    for (int32_t i = 0; i < n; ++i) {
        int32_t s = slots[i];
        if (seq_len_[s] % page_size_ == 0) {
            int32_t p = take_lowest();
            size_t idx = static_cast<size_t>(s) * max_pages_ + seq_len_[s] / page_size_;
            table_[idx] = p;
            if (updates) { updates->push_back(static_cast<int32_t>(idx)); updates->push_back(p); }
        }
        seq_len_[s] += 1;
    }
    return OUTLETS_OK;
}

int Pager::release(int32_t n, const int32_t* slots, const char** why) {
    int rc = check_slots(n, slots, why);
    if (rc != OUTLETS_OK) return rc;
    for (int32_t i = 0; i < n; ++i) {
        int32_t s = slots[i];
        int32_t np = (seq_len_[s] + page_size_ - 1) / page_size_;
        for (int32_t j = 0; j < np; ++j) {
            size_t idx = static_cast<size_t>(s) * max_pages_ + j;
            free_.push(table_[idx]);
            table_[idx] = -1;
        }
        seq_len_[s] = 0;
    }
    return OUTLETS_OK;
}

int varlen_meta(int32_t n, const int32_t* lens, int32_t* cu, int32_t* pos, int32_t* last) {
    int64_t off = 0;
    if (cu) cu[0] = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (lens[i] <= 0) return OUTLETS_ERR_INVALID_ARG;
        if (pos)
            for (int32_t j = 0; j < lens[i]; ++j) pos[off + j] = j;
        off += lens[i];
        if (off > INT32_MAX) return OUTLETS_ERR_INVALID_ARG;
        if (cu) cu[i + 1] = static_cast<int32_t>(off);
        if (last) last[i] = static_cast<int32_t>(off - 1);
    }
    return OUTLETS_OK;
}

}  // namespace outlets
