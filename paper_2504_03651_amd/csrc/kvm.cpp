// kvm.cpp -- task-aware KV block manager (include/echo_kvm.h), host only.
//
// Section 4.2 (priority-based eviction, reference counts, the threshold for
// active requests) on top of prefix caching as described in Section 6: a
// free table ordered by (priority, last access time) from which the lowest
// entry is evicted when a block is needed and the empty set is exhausted.
#include <algorithm>
#include <array>
#include <cstring>
#include <new>
#include <set>
#include <unordered_map>
#include <vector>

#include "echo_kvm.h"
#include "status.hpp"

namespace {

using echo::fail;

constexpr int kTok = 16;          // tokens per block
enum { kEmpty = 0, kHeld = 1, kCached = 2 };

// splitmix64 finaliser (Steele, Lea and Flood, "Fast splittable pseudorandom
// number generators", 2014) as the mixing step of the prefix-chain hash
uint64_t mix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// hash of a full block: its predecessor's hash (0 for the first block) and
// its 16 tokens
uint64_t chain_hash(uint64_t parent, const int32_t *tok) {
    uint64_t h = mix64(parent ^ 0xD6E8FEB86659FD93ull);
    for (int i = 0; i < kTok; ++i) h = mix64(h ^ (uint32_t)tok[i]);
    return h;
}

struct FreeKey {
    int32_t p2;       // twice the eviction priority
    int64_t lat;      // last access time
    int32_t negdepth; // deeper blocks first
    int32_t id;
    bool operator<(const FreeKey &o) const {
        if (p2 != o.p2) return p2 < o.p2;
        if (lat != o.lat) return lat < o.lat;
        if (negdepth != o.negdepth) return negdepth < o.negdepth;
        return id < o.id;
    }
};

struct Block {
    int32_t state = kEmpty;
    int32_t holders = 0;
    int32_t task = ECHO_TASK_OFFLINE;
    int64_t lat = 0;
    int32_t depth = 0;
    int32_t ntok = 0;
    std::array<int32_t, kTok> tok{};
    uint64_t parent = 0;    // hash of the preceding full block (0: first)
    uint64_t hash = 0;      // valid when hashed (the block is full)
    bool hashed = false;
    bool published = false; // the cache map points at this block
    FreeKey key{};          // valid when cached
};

struct Seq {
    int32_t task = ECHO_TASK_OFFLINE;
    int32_t len = 0;
    std::vector<int32_t> blocks;
};

}  // namespace

struct echo_kvm {
    int32_t nb = 0, limit = 0;
    int64_t now = 0;
    int32_t held = 0;
    int64_t hits_tokens = 0, evictions = 0;
    std::vector<Block> blk;
    std::set<int32_t> empty;
    std::set<FreeKey> freetab;
    std::unordered_map<uint64_t, int32_t> cache;   // published hash -> block
    std::unordered_map<uint64_t, int32_t> rc;      // hash -> registered offline prompts
    std::unordered_map<int64_t, std::vector<uint64_t>> reg;
    std::unordered_map<int64_t, Seq> seqs;
    std::vector<int32_t> pending;                  // filled blocks to publish at the tick
    std::vector<int32_t> copies;                   // queued (src, dst) pairs
    std::vector<int32_t> evicted;                  // queued evicted ids

    int32_t rc_of(const Block &b) const {
        if (!b.hashed) return 0;
        auto it = rc.find(b.hash);
        return it == rc.end() ? 0 : it->second;
    }
    int32_t prio2(const Block &b) const {
        const int32_t r = rc_of(b);
        if (r > 0) return 2 * r;
        return b.task == ECHO_TASK_ONLINE ? 1 : 0;
    }
    int32_t cached_reusable = 0;   // cached blocks with rc > 0
    void to_free(int32_t id) {
        Block &b = blk[id];
        b.state = kCached;
        b.key = FreeKey{prio2(b), b.lat, -b.depth, id};
        freetab.insert(b.key);
        cached_reusable += b.key.p2 >= 2;
    }
    void from_free(int32_t id) {
        freetab.erase(blk[id].key);
        cached_reusable -= blk[id].key.p2 >= 2;
    }
    void rekey(uint64_t h) {
        auto it = cache.find(h);
        if (it == cache.end()) return;
        Block &b = blk[it->second];
        if (b.state != kCached) return;
        from_free(it->second);
        to_free(it->second);
    }
    void reset(Block &b) { b = Block{}; }
    // a block for new content: the lowest empty id, else evict
    int32_t take() {
        int32_t id;
        if (!empty.empty()) {
            id = *empty.begin();
            empty.erase(empty.begin());
        } else {
            id = freetab.begin()->id;
            from_free(id);
            Block &b = blk[id];
            auto it = cache.find(b.hash);
            if (it != cache.end() && it->second == id) cache.erase(it);
            evicted.push_back(id);
            ++evictions;
        }
        Block &b = blk[id];
        reset(b);
        b.state = kHeld;
        b.holders = 1;
        ++held;
        return id;
    }
    void stamp(Block &b, int32_t task, int32_t depth) {
        b.lat = now;
        b.task = task;
        b.depth = depth;
    }
    void publish(int32_t id) {
        Block &b = blk[id];
        if (!b.hashed || b.published) return;
        if (cache.count(b.hash)) return;   // the same prefix is already cached elsewhere
        cache.emplace(b.hash, id);
        b.published = true;
    }
    // the published block holding exactly this prefix, or -1
    int32_t lookup(uint64_t parent, uint64_t h, const int32_t *tok) const {
        auto it = cache.find(h);
        if (it == cache.end()) return -1;
        const Block &b = blk[it->second];
        if (b.parent != parent || std::memcmp(b.tok.data(), tok, sizeof(int32_t) * kTok) != 0)
            return -1;
        return it->second;
    }
    int32_t available() const { return (int32_t)(empty.size() + freetab.size()); }
};

namespace {

int check_tokens(const int32_t *tokens, int32_t n, int32_t min_n) {
    if (n < min_n) return fail(ECHO_E_INVALID, "%d tokens (at least %d)", n, min_n);
    if (n > 0 && !tokens) return fail(ECHO_E_INVALID, "tokens is NULL");
    return ECHO_OK;
}

}  // namespace

extern "C" {

int echo_kvm_create(int32_t num_blocks, int32_t offline_limit, echo_kvm_t **out) {
    echo::clear_error();
    if (!out) return fail(ECHO_E_INVALID, "out is NULL");
    *out = nullptr;
    if (num_blocks <= 0 || offline_limit < 0 || offline_limit > num_blocks)
        return fail(ECHO_E_INVALID, "num_blocks %d, offline_limit %d", num_blocks, offline_limit);
    echo_kvm_t *m = new (std::nothrow) echo_kvm_t();
    if (!m) return fail(ECHO_E_INVALID, "out of host memory");
    m->nb = num_blocks;
    m->limit = offline_limit;
    m->blk.resize((size_t)num_blocks);
    for (int32_t i = 0; i < num_blocks; ++i) m->empty.insert(m->empty.end(), i);
    *out = m;
    return ECHO_OK;
}

void echo_kvm_destroy(echo_kvm_t *m) { delete m; }

int echo_kvm_register_offline(echo_kvm_t *m, int64_t req, const int32_t *tokens, int32_t n) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    int rc = check_tokens(tokens, n, 0);
    if (rc) return rc;
    if (m->reg.count(req)) return fail(ECHO_E_INVALID, "request %lld already registered", (long long)req);
    std::vector<uint64_t> chain;
    uint64_t parent = 0;
    for (int32_t j = 0; j + kTok <= n; j += kTok) {
        parent = chain_hash(parent, tokens + j);
        chain.push_back(parent);
    }
    for (uint64_t h : chain) {
        ++m->rc[h];
        m->rekey(h);
    }
    m->reg.emplace(req, std::move(chain));
    return ECHO_OK;
}

int echo_kvm_unregister_offline(echo_kvm_t *m, int64_t req) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    auto it = m->reg.find(req);
    if (it == m->reg.end()) return fail(ECHO_E_INVALID, "request %lld not registered", (long long)req);
    for (uint64_t h : it->second) {
        auto r = m->rc.find(h);
        if (--r->second == 0) m->rc.erase(r);
        m->rekey(h);
    }
    m->reg.erase(it);
    return ECHO_OK;
}

int echo_kvm_start(echo_kvm_t *m, int64_t seq, int32_t task, const int32_t *tokens, int32_t n,
                   int32_t *cached_tokens) {
    echo::clear_error();
    if (!m || !cached_tokens) return fail(ECHO_E_INVALID, "manager or cached_tokens is NULL");
    int rc = check_tokens(tokens, n, 1);
    if (rc) return rc;
    if (task != ECHO_TASK_ONLINE && task != ECHO_TASK_OFFLINE)
        return fail(ECHO_E_INVALID, "task %d", task);
    if (m->seqs.count(seq)) return fail(ECHO_E_INVALID, "sequence %lld is running", (long long)seq);
    const int32_t nfull = n / kTok, nblocks = (n + kTok - 1) / kTok;
    // leading full blocks already cached (prefix chain)
    std::vector<uint64_t> h((size_t)nfull);
    std::vector<int32_t> hits;
    uint64_t parent = 0;
    bool chain_open = true;
    for (int32_t j = 0; j < nfull; ++j) {
        h[j] = chain_hash(parent, tokens + (size_t)j * kTok);
        if (chain_open) {
            const int32_t b = m->lookup(parent, h[j], tokens + (size_t)j * kTok);
            if (b >= 0) hits.push_back(b);
            else chain_open = false;
        }
        parent = h[j];
    }
    if ((int32_t)hits.size() == nfull && n % kTok == 0 && !hits.empty()) hits.pop_back();
    const int32_t nhit = (int32_t)hits.size();
    int32_t from_free = 0;
    for (int32_t b : hits) from_free += m->blk[b].state == kCached;
    const int32_t n_new = nblocks - nhit;
    if (n_new > m->available() - from_free)
        return fail(ECHO_E_NOSPACE, "sequence %lld needs %d new blocks, %d available",
                    (long long)seq, n_new, m->available() - from_free);
    if (task == ECHO_TASK_OFFLINE && m->held + from_free + n_new > m->limit)
        return fail(ECHO_E_NOSPACE, "offline sequence %lld would hold %d blocks (limit %d)",
                    (long long)seq, m->held + from_free + n_new, m->limit);

    Seq s;
    s.task = task;
    s.len = n;
    for (int32_t j = 0; j < nhit; ++j) {
        const int32_t b = hits[j];
        Block &bk = m->blk[b];
        if (bk.state == kCached) {
            m->from_free(b);
            bk.state = kHeld;
            ++m->held;
        }
        ++bk.holders;
        m->stamp(bk, task, j);
        s.blocks.push_back(b);
    }
    for (int32_t j = nhit; j < nblocks; ++j) {
        const int32_t b = m->take();
        Block &bk = m->blk[b];
        bk.ntok = std::min(kTok, n - j * kTok);
        std::memcpy(bk.tok.data(), tokens + (size_t)j * kTok, sizeof(int32_t) * bk.ntok);
        bk.parent = j > 0 ? h[j - 1] : 0;
        if (j < nfull) {
            bk.hash = h[j];
            bk.hashed = true;
            m->pending.push_back(b);
        }
        m->stamp(bk, task, j);
        s.blocks.push_back(b);
    }
    m->seqs.emplace(seq, std::move(s));
    *cached_tokens = nhit * kTok;
    m->hits_tokens += nhit * kTok;
    return ECHO_OK;
}

int echo_kvm_probe(const echo_kvm_t *m, const int32_t *tokens, int32_t n, int32_t *cached_tokens) {
    echo::clear_error();
    if (!m || !cached_tokens) return fail(ECHO_E_INVALID, "manager or cached_tokens is NULL");
    int rc = check_tokens(tokens, n, 1);
    if (rc) return rc;
    const int32_t nfull = n / kTok;
    int32_t hits = 0;
    uint64_t parent = 0;
    for (int32_t j = 0; j < nfull; ++j) {
        const uint64_t h = chain_hash(parent, tokens + (size_t)j * kTok);
        if (m->lookup(parent, h, tokens + (size_t)j * kTok) < 0) break;
        ++hits;
        parent = h;
    }
    if (hits == nfull && n % kTok == 0 && hits > 0) --hits;
    *cached_tokens = hits * kTok;
    return ECHO_OK;
}

int echo_kvm_set_offline_limit(echo_kvm_t *m, int32_t offline_limit) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    if (offline_limit < 0 || offline_limit > m->nb)
        return fail(ECHO_E_INVALID, "offline_limit %d of %d blocks", offline_limit, m->nb);
    m->limit = offline_limit;
    return ECHO_OK;
}

int echo_kvm_append(echo_kvm_t *m, int64_t seq, const int32_t *tokens, int32_t n) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    int rc = check_tokens(tokens, n, 1);
    if (rc) return rc;
    auto it = m->seqs.find(seq);
    if (it == m->seqs.end()) return fail(ECHO_E_INVALID, "sequence %lld is not running", (long long)seq);
    Seq &s = it->second;
    const bool cow = s.len % kTok != 0 && m->blk[s.blocks.back()].holders > 1;
    const int32_t n_new = (s.len + n + kTok - 1) / kTok - (int32_t)s.blocks.size() + (cow ? 1 : 0);
    if (n_new > m->available())
        return fail(ECHO_E_NOSPACE, "sequence %lld needs %d new blocks, %d available",
                    (long long)seq, n_new, m->available());
    if (s.task == ECHO_TASK_OFFLINE && n_new > 0 && m->held + n_new > m->limit)
        return fail(ECHO_E_NOSPACE, "offline sequence %lld would hold %d blocks (limit %d)",
                    (long long)seq, m->held + n_new, m->limit);
    if (cow) {
        const int32_t src = s.blocks.back();
        const int32_t dst = m->take();
        Block &d = m->blk[dst];
        const Block &sb = m->blk[src];
        d.ntok = sb.ntok;
        d.tok = sb.tok;
        d.parent = sb.parent;
        --m->blk[src].holders;
        s.blocks.back() = dst;
        m->copies.push_back(src);
        m->copies.push_back(dst);
    }
    for (int32_t i = 0; i < n; ++i) {
        if (s.len % kTok == 0) {
            const int32_t b = m->take();
            const int32_t j = (int32_t)s.blocks.size();
            m->blk[b].parent = j > 0 ? m->blk[s.blocks[j - 1]].hash : 0;
            s.blocks.push_back(b);
        }
        const int32_t j = (int32_t)s.blocks.size() - 1;
        Block &bk = m->blk[s.blocks[j]];
        bk.tok[bk.ntok++] = tokens[i];
        ++s.len;
        m->stamp(bk, s.task, j);
        if (bk.ntok == kTok) {
            bk.hash = chain_hash(bk.parent, bk.tok.data());
            bk.hashed = true;
            m->pending.push_back(s.blocks[j]);
        }
    }
    return ECHO_OK;
}

int echo_kvm_fork(echo_kvm_t *m, int64_t parent, int64_t child) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    auto it = m->seqs.find(parent);
    if (it == m->seqs.end()) return fail(ECHO_E_INVALID, "sequence %lld is not running", (long long)parent);
    if (m->seqs.count(child)) return fail(ECHO_E_INVALID, "sequence %lld is running", (long long)child);
    Seq c = it->second;
    for (size_t j = 0; j < c.blocks.size(); ++j) {
        Block &bk = m->blk[c.blocks[j]];
        ++bk.holders;
        m->stamp(bk, c.task, (int32_t)j);
    }
    m->seqs.emplace(child, std::move(c));
    return ECHO_OK;
}

int echo_kvm_finish(echo_kvm_t *m, int64_t seq) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    auto it = m->seqs.find(seq);
    if (it == m->seqs.end()) return fail(ECHO_E_INVALID, "sequence %lld is not running", (long long)seq);
    const Seq &s = it->second;
    for (int32_t b : s.blocks) m->publish(b);
    for (int32_t j = (int32_t)s.blocks.size() - 1; j >= 0; --j) {
        const int32_t b = s.blocks[j];
        Block &bk = m->blk[b];
        m->stamp(bk, s.task, j);
        if (--bk.holders > 0) continue;
        --m->held;
        if (bk.published) {
            m->to_free(b);
        } else {
            m->reset(bk);
            m->empty.insert(b);
        }
    }
    m->seqs.erase(it);
    return ECHO_OK;
}

int echo_kvm_tick(echo_kvm_t *m) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    for (int32_t b : m->pending) m->publish(b);
    m->pending.clear();
    ++m->now;
    return ECHO_OK;
}

int echo_kvm_block_tables(const echo_kvm_t *m, const int64_t *seqs, int32_t rows,
                          int32_t max_blocks_per_row, int32_t *block_tables, int32_t *seq_lens) {
    echo::clear_error();
    if (!m) return fail(ECHO_E_INVALID, "manager is NULL");
    if (rows < 0 || max_blocks_per_row <= 0) return fail(ECHO_E_INVALID, "rows %d, max_blocks_per_row %d", rows, max_blocks_per_row);
    if (rows > 0 && (!seqs || !block_tables || !seq_lens)) return fail(ECHO_E_INVALID, "NULL array");
    for (int32_t r = 0; r < rows; ++r) {
        auto it = m->seqs.find(seqs[r]);
        if (it == m->seqs.end())
            return fail(ECHO_E_INVALID, "row %d: sequence %lld is not running", r, (long long)seqs[r]);
        if ((int32_t)it->second.blocks.size() > max_blocks_per_row)
            return fail(ECHO_E_RANGE, "row %d holds %zu blocks, rows hold %d", r,
                        it->second.blocks.size(), max_blocks_per_row);
    }
    for (int32_t r = 0; r < rows; ++r) {
        const Seq &s = m->seqs.find(seqs[r])->second;
        int32_t *row = block_tables + (size_t)r * max_blocks_per_row;
        for (int32_t j = 0; j < max_blocks_per_row; ++j)
            row[j] = j < (int32_t)s.blocks.size() ? s.blocks[j] : -1;
        seq_lens[r] = s.len;
    }
    return ECHO_OK;
}

int echo_kvm_take_copies(echo_kvm_t *m, int32_t *pairs, int32_t max_pairs, int32_t *n_pairs) {
    echo::clear_error();
    if (!m || !n_pairs || max_pairs < 0 || (max_pairs > 0 && !pairs))
        return fail(ECHO_E_INVALID, "bad arguments");
    const int32_t k = std::min<int32_t>(max_pairs, (int32_t)(m->copies.size() / 2));
    if (k > 0) std::memcpy(pairs, m->copies.data(), sizeof(int32_t) * 2 * k);
    m->copies.erase(m->copies.begin(), m->copies.begin() + 2 * k);
    *n_pairs = k;
    return ECHO_OK;
}

int echo_kvm_take_evictions(echo_kvm_t *m, int32_t *blocks, int32_t max, int32_t *n) {
    echo::clear_error();
    if (!m || !n || max < 0 || (max > 0 && !blocks)) return fail(ECHO_E_INVALID, "bad arguments");
    const int32_t k = std::min<int32_t>(max, (int32_t)m->evicted.size());
    if (k > 0) std::memcpy(blocks, m->evicted.data(), sizeof(int32_t) * k);
    m->evicted.erase(m->evicted.begin(), m->evicted.begin() + k);
    *n = k;
    return ECHO_OK;
}

int echo_kvm_block_info(const echo_kvm_t *m, int32_t block, echo_kvm_block_info_t *info) {
    echo::clear_error();
    if (!m || !info) return fail(ECHO_E_INVALID, "manager or info is NULL");
    if (block < 0 || block >= m->nb) return fail(ECHO_E_RANGE, "block %d of %d", block, m->nb);
    const Block &b = m->blk[block];
    info->state = b.state;
    info->holders = b.holders;
    info->rc = m->rc_of(b);
    info->task = b.task;
    info->lat = b.lat;
    info->priority2 = b.state == kCached ? b.key.p2 : -1;
    info->depth = b.depth;
    return ECHO_OK;
}

int echo_kvm_stats(const echo_kvm_t *m, echo_kvm_stats_t *st) {
    echo::clear_error();
    if (!m || !st) return fail(ECHO_E_INVALID, "manager or stats is NULL");
    st->empty = (int32_t)m->empty.size();
    st->held = m->held;
    st->cached = (int32_t)m->freetab.size();
    st->running = (int32_t)m->seqs.size();
    st->now = m->now;
    st->hits_tokens = m->hits_tokens;
    st->evictions = m->evictions;
    st->cached_reusable = m->cached_reusable;
    return ECHO_OK;
}

}  // extern "C"
