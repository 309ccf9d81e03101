// Host-side paged-KV block manager (Table 1, "KV manager").
//
// Blocks of 16 positions; a sequence grows by whole blocks taking the
// lowest-numbered free block first; a group of reservations is all or nothing.
#pragma once

#include <cstdint>
#include <functional>
#include <queue>
#include <unordered_map>
#include <utility>
#include <vector>

namespace slw {

class KvManager {
public:
    void reset(int32_t num_blocks, int32_t block_size);
    int32_t num_blocks() const { return num_blocks_; }
    int32_t block_size() const { return block_size_; }
    int32_t free_count() const { return static_cast<int32_t>(free_.size()); }

    bool exists(int64_t id) const { return seqs_.count(id) != 0; }
    // Each returns an SLW_* code (and sets the error message on failure).
    int create(int64_t id);
    int release(int64_t id);
    // What a reservation changed: per grown sequence, its block count and
    // reserved length before the call.
    struct Undo {
        struct Entry {
            int64_t id;
            size_t blocks;
            int32_t reserved;
        };
        std::vector<Entry> grown;
    };
    // Grows every (id, new_len) in order; all or nothing.  With `undo`, the
    // changes are recorded so that rollback() can return them.
    int reserve_all(const std::vector<std::pair<int64_t, int32_t>>& req, Undo* undo = nullptr);
    // Returns the blocks a reservation took and restores the lengths; the
    // free set, and so every later allocation, is as before the reservation.
    void rollback(const Undo& undo);

    const std::vector<int32_t>& table(int64_t id) const { return seqs_.at(id).blocks; }
    int32_t reserved(int64_t id) const { return seqs_.at(id).reserved; }
    int32_t slot(int64_t id, int32_t pos) const {
        const auto& bt = seqs_.at(id).blocks;
        return bt[pos / block_size_] * block_size_ + pos % block_size_;
    }

private:
    struct Seq {
        std::vector<int32_t> blocks;
        int32_t reserved = 0;
    };
    int32_t num_blocks_ = 0;
    int32_t block_size_ = 16;
    std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> free_;
    std::unordered_map<int64_t, Seq> seqs_;
};

}  // namespace slw
