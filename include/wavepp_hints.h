/*
 * wavepp_hints.h -- C ABI of the reuse-hint machinery in libwavepp_attn.so: chained block hashes,
 * a sharded counted hint index, and the probes that turn a request's block keys into a reusable
 * endpoint.  Host only: no HIP call.
 *
 * Behaviour (Design of WavePP, "Fast Reuse Hints"):
 *   - Chained prefix hash over full token blocks (Eq. 5): H_{-1} = 0,
 *     H_i = hash(B_i, extraKeys_i, salt, H_{i-1}).  The paper leaves the hash open; here it is
 *     SHA-256 (FIPS 180-4) of  salt || H_{i-1} (32 bytes) || extraKeys_i (int64 LE each) ||
 *     B_i (int32 tokens, LE), with H_{-1} = 32 zero bytes.  The index key of a block is the first
 *     8 bytes of H_i read as a little-endian uint64.  A trailing partial block is not hashed.
 *   - The index holds no blocks: a counter per (window, key), incremented when a block enters the
 *     cache tree and decremented when it is detached; the entry disappears at zero.  Offloading a
 *     block does not change it.  Keys are spread over shards, each with its own mutex; every probe
 *     takes only the mutex of the shard it reads, so the view may change during a lookup (it is a
 *     hint; an authoritative walk validates it later).
 *   - Dense-prefix probe: the number of leading blocks whose keys are all present, found by probing
 *     depths 1, 2, 4, ... until the first miss and bisecting between the last hit and that miss:
 *     O(log N) probes.  It equals the plain scan whenever the indexed keys are prefix-closed, as a
 *     cache tree's are.
 *   - Recurrent probe: from a limit, the scan goes backwards to the nearest boundary j with a
 *     snapshot (the snapshot at boundary j is indexed under block j - 1's key); 0 if none.
 *
 * Thread safety: the index may be used from several threads at once; a probe sees each key as of
 * the moment its shard was read.
 * Errors: wavepp_status codes (wavepp_attn.h), details in wavepp_last_error().
 */
#ifndef WAVEPP_HINTS_H
#define WAVEPP_HINTS_H

#include "wavepp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Chained hashes of the floor(n_tokens / block) full blocks of `tokens`.  extra_keys is NULL or
 * [n_blocks][extra_per_block] int64; salt may be NULL when salt_len = 0.  Writes 32 bytes per
 * block to `digests` (may be NULL) and the block's index key to `keys` (may be NULL).  Returns the
 * number of blocks, or a negative status. */
int64_t wavepp_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block, const int64_t* extra_keys,
                            int32_t extra_per_block, const uint8_t* salt, int32_t salt_len, uint8_t* digests,
                            uint64_t* keys);

typedef struct wavepp_hint_index_s wavepp_hint_index_t;

int wavepp_hint_index_create(int32_t num_shards, wavepp_hint_index_t** out);

/* A block of `window` entered the cache tree: +1 on each key. */
int wavepp_hint_index_add(wavepp_hint_index_t* index, int32_t window, const uint64_t* keys, int64_t n);

/* A block was detached from the tree: -1 on each key, erased at 0.  A key that is not present is
 * an error (WAVEPP_EINVAL); the keys before it in the array have been detached. */
int wavepp_hint_index_detach(wavepp_hint_index_t* index, int32_t window, const uint64_t* keys, int64_t n);

/* Entries (distinct (window, key) pairs) currently indexed. */
int64_t wavepp_hint_index_size(wavepp_hint_index_t* index);

/* Dense-prefix endpoint by gallop and bisect.  *probes receives the number of keys looked up. */
int wavepp_hint_probe_prefix(wavepp_hint_index_t* index, int32_t window, const uint64_t* keys, int64_t n,
                             int64_t* endpoint, int32_t* probes);

/* The same endpoint by the plain scan from the first block (O(N) probes), for comparison. */
int wavepp_hint_probe_prefix_linear(wavepp_hint_index_t* index, int32_t window, const uint64_t* keys, int64_t n,
                                    int64_t* endpoint, int32_t* probes);

/* Largest boundary j <= limit (limit <= number of keys) with a snapshot, scanning backwards. */
int wavepp_hint_probe_recurrent(wavepp_hint_index_t* index, int32_t window, const uint64_t* keys, int64_t limit,
                                int64_t* endpoint, int32_t* probes);

void wavepp_hint_index_destroy(wavepp_hint_index_t* index);

#ifdef __cplusplus
}
#endif

#endif /* WAVEPP_HINTS_H */
