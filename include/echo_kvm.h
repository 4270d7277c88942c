/*
 * echo_kvm.h -- task-aware KV block manager (host only, no GPU work).
 *
 * Keeps the paged KV cache's block bookkeeping for online (latency-bound) and
 * offline (throughput) sequences and emits what the iteration entry points of
 * echo.h consume: per-row block tables and sequence lengths, and the
 * (src, dst) pairs that echo_block_copy must copy before an append
 * (copy-on-write).  It follows Section 4.2 ("KV Cache Manager") and the KV
 * cache manager of Section 6 (automatic prefix caching extended with
 * task-aware eviction priorities):
 *
 *   - Blocks of 16 tokens.  A full block is identified by its whole token
 *     prefix; a later sequence whose prompt starts with the same full blocks
 *     reuses them (prefix caching).  Partial blocks are private.
 *   - A block referenced by a running sequence ("held") is never evicted.
 *     A released full block stays cached in a free table until it is needed
 *     for another block; blocks are evicted lowest priority first:
 *         rc > 0                     priority rc  (rc = registered offline
 *                                    requests whose prompt contains the
 *                                    block's prefix, the running one included)
 *         last used by online task   priority 1/2
 *         last used by offline task  priority 0
 *     and, within a priority, least recently used first (last access time),
 *     then the block deeper in its sequence first, then the lower block id.
 *     Blocks that were never filled or are partial go straight back to the
 *     empty set, which is always used before anything is evicted (lowest id
 *     first).
 *   - Threshold: blocks held by running sequences may exceed `offline_limit`
 *     only through online sequences; an offline start or append that would
 *     take more held blocks than the limit fails with ECHO_E_NOSPACE, so the
 *     rest of the pool stays for bursts of online requests.
 *
 * Time: every call stamps the blocks it touches with the manager's clock;
 * echo_kvm_tick() ends an iteration, advances the clock and makes the full
 * blocks filled during that iteration visible to prefix lookups (their KV is
 * written by the iteration's append).  echo_kvm_finish() does the same for the
 * finishing sequence's blocks.
 *
 * Every call validates first and changes nothing when it fails.  A manager is
 * not thread-safe: one thread (the scheduler) owns it.
 */
#ifndef ECHO_KVM_H
#define ECHO_KVM_H

#include <stddef.h>
#include <stdint.h>

#include "echo.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct echo_kvm echo_kvm_t;

typedef enum { ECHO_TASK_ONLINE = 0, ECHO_TASK_OFFLINE = 1 } echo_task_t;

/* A manager of num_blocks blocks (> 0); offline_limit (0..num_blocks) caps the
 * held blocks that offline starts and appends may reach.  *out receives the
 * manager (ECHO_E_INVALID on bad sizes). */
int echo_kvm_create(int32_t num_blocks, int32_t offline_limit, echo_kvm_t **out);
void echo_kvm_destroy(echo_kvm_t *m);

/* Reference counts: an offline request registers its prompt (host tokens,
 * n >= 0) when it enters the offline pool and unregisters when it completes
 * or is dropped; every full block of the prompt's prefix chain counts it.
 * ECHO_E_INVALID for an id registered twice or unknown. */
int echo_kvm_register_offline(echo_kvm_t *m, int64_t req, const int32_t *tokens, int32_t n);
int echo_kvm_unregister_offline(echo_kvm_t *m, int64_t req);

/* Starts sequence `seq` (not running) of task ECHO_TASK_* with its prompt
 * tokens[0..n), n >= 1.  Leading full blocks found in the cache are reused and
 * *cached_tokens (16 per reused block) tells how many prompt tokens already
 * have KV; the prompt's last full block is never reused when it would leave no
 * token to compute, so *cached_tokens < n.  The remaining blocks are taken
 * from the empty set, then by eviction.  ECHO_E_NOSPACE when they do not fit
 * (or, offline, the limit). */
int echo_kvm_start(echo_kvm_t *m, int64_t seq, int32_t task, const int32_t *tokens, int32_t n,
                   int32_t *cached_tokens);

/* How many prompt tokens echo_kvm_start would find cached for tokens[0..n)
 * (n >= 1), in *cached_tokens, without changing anything. */
int echo_kvm_probe(const echo_kvm_t *m, const int32_t *tokens, int32_t n, int32_t *cached_tokens);

/* Moves the threshold (0..num_blocks): later offline starts and appends may
 * not raise the held blocks above it; blocks already held stay. */
int echo_kvm_set_offline_limit(echo_kvm_t *m, int32_t offline_limit);

/* Appends tokens[0..n) (n >= 1) to running sequence `seq`.  When its last
 * block is partial and shared (after echo_kvm_fork), the block is copied into
 * a new private one first and the pair is queued for echo_kvm_take_copies. */
int echo_kvm_append(echo_kvm_t *m, int64_t seq, const int32_t *tokens, int32_t n);

/* Starts `child` (not running) as a copy of running `parent` sharing all its
 * blocks (parallel sampling). */
int echo_kvm_fork(echo_kvm_t *m, int64_t parent, int64_t child);

/* Ends running sequence `seq` (completed, or preempted to be recomputed
 * later): its blocks are released to the free table or the empty set. */
int echo_kvm_finish(echo_kvm_t *m, int64_t seq);

/* Ends an iteration (see Time above). */
int echo_kvm_tick(echo_kvm_t *m);

/* Block tables of `rows` running sequences, in order: block_tables
 * [rows][max_blocks_per_row] (unused entries -1) and seq_lens [rows], host
 * memory.  ECHO_E_RANGE when a sequence has more blocks than a row holds. */
int echo_kvm_block_tables(const echo_kvm_t *m, const int64_t *seqs, int32_t rows,
                          int32_t max_blocks_per_row, int32_t *block_tables, int32_t *seq_lens);

/* Moves the queued copy-on-write pairs (src, dst) into pairs[2 * k] (at most
 * max_pairs) and sets *n_pairs; pairs that do not fit stay queued. */
int echo_kvm_take_copies(echo_kvm_t *m, int32_t *pairs, int32_t max_pairs, int32_t *n_pairs);

/* Moves the ids of blocks evicted since the last call (in eviction order,
 * at most max) into blocks and sets *n; the rest stay queued. */
int echo_kvm_take_evictions(echo_kvm_t *m, int32_t *blocks, int32_t max, int32_t *n);

typedef struct {
    int32_t state;      /* 0 empty, 1 held, 2 cached (evictable) */
    int32_t holders;    /* running sequences referencing the block */
    int32_t rc;         /* registered offline prompts containing its prefix */
    int32_t task;       /* task of the last access */
    int64_t lat;        /* last access time */
    int32_t priority2;  /* twice the eviction priority (cached blocks) */
    int32_t depth;      /* block index in the sequence of its last access */
} echo_kvm_block_info_t;

int echo_kvm_block_info(const echo_kvm_t *m, int32_t block, echo_kvm_block_info_t *info);

typedef struct {
    int32_t empty, held, cached;  /* blocks per state */
    int32_t running;              /* running sequences */
    int64_t now;                  /* clock */
    int64_t hits_tokens;          /* prompt tokens served from the cache so far */
    int64_t evictions;            /* blocks evicted so far */
    int32_t cached_reusable;      /* cached blocks with rc > 0 (evicting them costs recompute) */
} echo_kvm_stats_t;

int echo_kvm_stats(const echo_kvm_t *m, echo_kvm_stats_t *stats);

#ifdef __cplusplus
}
#endif

#endif /* ECHO_KVM_H */
