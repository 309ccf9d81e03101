// Host-side paged-KV block manager (Table 1, "KV manager").
#include "kv_manager.h"

#include <unordered_map>

#include "common.h"

namespace slw {

void KvManager::reset(int32_t num_blocks, int32_t block_size) {
    num_blocks_ = num_blocks;
    block_size_ = block_size;
    seqs_.clear();
    std::vector<int32_t> ids(num_blocks);
    for (int32_t i = 0; i < num_blocks; ++i) ids[i] = i;
    free_ = decltype(free_)(std::greater<int32_t>(), std::move(ids));
}

int KvManager::create(int64_t id) {
    if (seqs_.count(id)) return fail(SLW_EINVAL, "sequence %lld already exists", (long long)id);
    seqs_.emplace(id, Seq{});
    return SLW_OK;
}

int KvManager::release(int64_t id) {
    auto it = seqs_.find(id);
    if (it == seqs_.end()) return fail(SLW_EINVAL, "sequence %lld unknown", (long long)id);
    for (int32_t b : it->second.blocks) free_.push(b);
    seqs_.erase(it);
    return SLW_OK;
}

int KvManager::reserve_all(const std::vector<std::pair<int64_t, int32_t>>& req, Undo* undo) {
    if (undo) undo->grown.clear();
    // Largest request per sequence, then the total number of new blocks.
    std::unordered_map<int64_t, int32_t> want;
    for (const auto& r : req) {
        auto it = seqs_.find(r.first);
        if (it == seqs_.end()) return fail(SLW_EINVAL, "sequence %lld unknown", (long long)r.first);
        if (r.second < 0) return fail(SLW_EINVAL, "negative length for sequence %lld", (long long)r.first);
        auto w = want.find(r.first);
        if (w == want.end()) want.emplace(r.first, r.second);
        else if (r.second > w->second) w->second = r.second;
    }
    int64_t total = 0;
    for (const auto& w : want) {
        const Seq& s = seqs_.at(w.first);
        int64_t len = w.second > s.reserved ? w.second : s.reserved;
        int64_t need = ceil_div(len, block_size_) - static_cast<int64_t>(s.blocks.size());
        if (need > 0) total += need;
    }
    if (total > static_cast<int64_t>(free_.size()))
        return fail(SLW_ENOMEM, "KV pool exhausted: need %lld blocks, %d free", (long long)total,
                    free_count());
    // Grow in request order so block ids are deterministic.
    for (const auto& r : req) {
        auto w = want.find(r.first);
        if (w == want.end()) continue;  // already grown
        Seq& s = seqs_.at(r.first);
        int32_t len = w->second > s.reserved ? w->second : s.reserved;
        int64_t need = ceil_div(len, block_size_) - static_cast<int64_t>(s.blocks.size());
        if (undo) undo->grown.push_back({r.first, s.blocks.size(), s.reserved});
        for (int64_t i = 0; i < need; ++i) {
            s.blocks.push_back(free_.top());
            free_.pop();
        }
        s.reserved = len;
        want.erase(w);
    }
    return SLW_OK;
}

void KvManager::rollback(const Undo& undo) {
    for (auto e = undo.grown.rbegin(); e != undo.grown.rend(); ++e) {
        Seq& s = seqs_.at(e->id);
        while (s.blocks.size() > e->blocks) {
            free_.push(s.blocks.back());
            s.blocks.pop_back();
        }
        s.reserved = e->reserved;
    }
}

}  // namespace slw
