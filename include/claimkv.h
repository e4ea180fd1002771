/*
 * claimkv.h -- C ABI of the claim-scoped KV materialization checker for
 * MI355X (gfx950).
 *
 * What it implements.  The paper ("Fail-Closed Lowering of Resident KV
 * Claims onto LLM Serving Runtimes", arXiv 2606.01387) requires an
 * offloadable claim to carry a stable identity, explicit acceptance before
 * offload, a materialization predicate, restoration before reuse and a
 * claim-scoped restoration-failure outcome, with ordered lifecycle events
 * (section 1 running example; Table 1; section 3 offloadable bundle;
 * section 7 event list and witness paths A, B, C).  Ambiguity must fail
 * closed (Table 2, last rule).  This library supplies those obligations for
 * paged KV blocks on the GPU:
 *
 *   claim_offload  accept a claim batch; each claim keeps its own offload
 *                  record, a 64-bit digest of every block it references
 *                  (optionally staging the bytes);
 *   claim_restore  move accepted, offloaded claims to restore-required,
 *                  optionally scattering staged bytes back, and apply the
 *                  given faults (bit flips = silent corruption, reported load
 *                  failures = the paper's controlled CPU->GPU load failure,
 *                  which fails the claims that recorded the block before it);
 *   claim_check    re-digest the referenced blocks, compare each claim's
 *                  blocks with its own offload record, chain each claim's
 *                  token prefix hash and reduce every claim to one
 *                  outcome (MATERIALIZED, RESTORE_FAILED_FAIL_CLOSED or
 *                  UNKNOWN) with the first failing block, appending the
 *                  ordered events;
 *   outcomes_read  copy the last check's outcomes and the new events to the
 *                  host;
 *   claim_lookup   the reuse lookup: how many leading token blocks of each
 *                  request hit the identities that offloads registered;
 *   claim_identity_stats  registered and ambiguous identities;
 *   claim_staging_reset   start a new generation of the staged bytes (the
 *                  offload tier), which staged offloads into one buffer
 *                  otherwise accumulate;
 *   claim_check_static    claim_check without any allocation, for callers
 *                  that cannot allocate (graph capture, serving loops);
 *   claim_digest_grid     the digest grid a launch takes.
 *
 * The digest, keys and chain are this library's definitions (the paper
 * leaves the byte-level check open; section 7 path B only requires
 * affected-block evidence for the failure):
 *   mix64(z)         SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014);
 *   splitmix64(x)    = mix64(x + 0x9E3779B97F4A7C15);
 *   splitmix64(s,i)  = mix64(s + (i+1) * 0x9E3779B97F4A7C15);
 *   k_i = splitmix64(S, i) | 1,  D(b) = sum_i w_i * k_i mod 2^64 over the
 *         little-endian 64-bit words w_i of block b's canonical bytes (the
 *         concatenation of its chunks, plane 0 first);
 *   t_m = splitmix64(~S, m) | 1, M_j = sum_m tok[j*bs+m] * t_m over the
 *         tokens present in token block j;
 *   h_{-1} = S,  h_j = splitmix64(h_{j-1} xor M_j).
 * S is the pool seed: with the block geometry it is the pool's cache
 * identity (Table 5, fixed cache identity).
 *
 * Conventions for every call:
 *   - all functions return a status (CLAIM_OK or a negative CLAIM_E*) and
 *     never abort;
 *   - argument, layout or size errors return CLAIM_EINVAL before any work is
 *     queued, and leave the pool unchanged;
 *   - per-claim problems are never errors: they become UNKNOWN outcomes;
 *   - work is queued on the pool's stream in call order; only
 *     claim_offload (for its acceptance verdict and to settle its counts),
 *     claim_restore (to read the host fault lists), outcomes_read,
 *     claim_block_state_read, claim_timing_read, claim_identity_stats and
 *     claim_pool_destroy wait for the stream, and claim_check waits, then
 *     allocates, only when its batch has more claims than any earlier call
 *     of the pool (the per-claim scratch grows to at least 1024 claims and
 *     is kept until claim_pool_destroy);
 *   - device arrays passed in a claim_batch must stay valid and unchanged
 *     until the queued work that reads them has completed;
 *   - calls on one pool must not overlap from several host threads.
 */
#ifndef CLAIMKV_H
#define CLAIMKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------- status */
#define CLAIM_OK 0
#define CLAIM_EINVAL (-1) /* bad argument, layout or size */
#define CLAIM_ENOMEM (-2) /* device allocation failed */
#define CLAIM_EHIP (-3)   /* HIP runtime error */
#define CLAIM_ENOSPC (-4) /* registry, footprint store, event log, staging or output too small */
#define CLAIM_EDUP (-5)   /* duplicate claim id: acceptance refused */
#define CLAIM_ELIMIT (-6) /* batch larger than claim_check_static's fixed scratch */

/* ----------------------------------------------------------- outcomes */
#define CLAIM_UNKNOWN 0 /* no claim outcome (ambiguity fails closed); zero-initialised = fail closed */
#define CLAIM_MATERIALIZED 1
#define CLAIM_RESTORE_FAILED_FAIL_CLOSED 2

/* ------------------------------------------------------- event kinds
 * Equivalent names are acceptable to the paper (section 4; section 7).
 * The section-7 events they stand for are given in brackets. */
#define CLAIM_EV_ACCEPTED 1               /* claim metadata accepted [E0] */
#define CLAIM_EV_OFFLOADED 2              /* whole footprint offloaded [E5] */
#define CLAIM_EV_RESTORE_REQUIRED 3       /* reuse requires restoration [E6] */
#define CLAIM_EV_RESTORED 4               /* restored and verified [E8] */
#define CLAIM_EV_RESTORATION_FAILED 5     /* claim-scoped failure [E11, E12] */
#define CLAIM_EV_ACTIVE_REQUEST_REFUSED 6 /* fail-closed refusal, blocking id [E13] */
#define CLAIM_EV_OUTCOME_UNKNOWN 7        /* no outcome: ambiguity (Table 3 unknown) */

/* ------------------------------------------- reason bits of an outcome */
#define CLAIM_R_NOT_ACCEPTED 0x001      /* id not registered */
#define CLAIM_R_NOT_OFFLOADED 0x002     /* registered, footprint not fully offloaded */
#define CLAIM_R_NO_RESTORE 0x004        /* no restore ordered before this check */
#define CLAIM_R_TOKEN_MISMATCH 0x008    /* token count, or a block's chain hash, differs from acceptance */
#define CLAIM_R_FOOTPRINT_MISMATCH 0x010 /* block list differs from acceptance */
#define CLAIM_R_MISSING_ENTRY 0x020     /* entry is CLAIM_NONE or >= num_blocks */
#define CLAIM_R_NO_OFFLOAD_RECORD 0x040 /* the claim recorded no offload of this block at this position */
#define CLAIM_R_SHAPE_MISMATCH 0x080    /* blocks != ceil(tokens / block_size) */
#define CLAIM_R_EMPTY 0x100             /* claim has no blocks */
#define CLAIM_R_MALFORMED 0x200         /* offsets inconsistent, or reserved id */
#define CLAIM_R_LOAD_FAILED 0x400       /* load failure reported after the claim's offload */
#define CLAIM_R_DIGEST_MISMATCH 0x800   /* restored digest != the claim's own offload digest */
#define CLAIM_R_BEYOND_PREDICATE 0x1000 /* a failed block lies past the predicate (not a failure) */

#define CLAIM_NONE 0xFFFFFFFFu                   /* no position; missing block-table entry */
#define CLAIM_RESERVED_ID 0xFFFFFFFFFFFFFFFFull /* never a valid claim id */

#define CLAIM_POOL_TIMING 0x1u       /* desc.flags: time the digest kernel of every claim_check */
#define CLAIM_POOL_STAGE_TIMING 0x2u /* desc.flags: also time every other stage (adds about 20 us per check) */

typedef struct claim_pool claim_pool;

/* Pool description.  The KV memory is caller-owned device memory laid out
 * [plane][block][chunk]: plane p = 2*layer + (0 for K, 1 for V) when
 * planes_per_layer = 2, p = layer for an MLA latent (planes_per_layer = 1);
 * a chunk is block_size x num_kv_heads x head_dim elements of elem_bytes
 * bytes in [token][head][dim] order, and must be a multiple of 16 bytes.
 * Element bytes are never interpreted (bf16 and fp8 are hashed as bytes).
 *
 * A pool may hold a head shard of every block, as one GPU does under tensor
 * parallelism by KV head: heads [first_kv_head, first_kv_head +
 * num_kv_heads) of blocks whose full width is total_kv_heads heads (its
 * chunks hold only its own heads, [token][head][dim] as above).  Each of its
 * 64-bit words keeps the key of its position in the full block's canonical
 * bytes, so a shard's block digest is the full digest's sum over the shard's
 * words, and the digests of a block's shards add up, mod 2^64, to the
 * digest of the whole block.  head_dim * elem_bytes must then be a multiple
 * of 8.  total_kv_heads = 0 (or num_kv_heads, with first_kv_head = 0) is a
 * pool of whole blocks; first_kv_head + num_kv_heads > total_kv_heads is
 * EINVAL. */
typedef struct claim_pool_desc {
  uint32_t num_layers;
  uint32_t planes_per_layer; /* 1 or 2 */
  uint32_t block_size;       /* tokens per block, 1..1024 */
  uint32_t num_kv_heads;
  uint32_t head_dim;
  uint32_t elem_bytes;
  uint32_t num_blocks;       /* < CLAIM_NONE */
  uint32_t flags;            /* CLAIM_POOL_TIMING | CLAIM_POOL_STAGE_TIMING */
  uint64_t seed;             /* cache-identity seed S */
  void* kv_base;             /* device pointer, 16-byte aligned */
  uint64_t kv_bytes;         /* >= planes * num_blocks * chunk bytes */
  void* stream;              /* hipStream_t (NULL = default stream) */
  uint64_t max_claims;       /* registry capacity (claims ever accepted) */
  uint64_t max_footprint;    /* block-table entries ever accepted */
  uint64_t event_capacity;   /* event records held between outcomes_read calls */
  uint32_t total_kv_heads;   /* head shard: KV heads of the full block (0: num_kv_heads) */
  uint32_t first_kv_head;    /* head shard: full-block index of this pool's first head */
} claim_pool_desc;

/* A claim batch in compressed rows.  All arrays are device memory owned by
 * the caller.  Claim c has block-table entries block_ids[block_offsets[c] ..
 * block_offsets[c+1]) (CLAIM_NONE = missing entry) and token ids
 * tokens[token_offsets[c] .. token_offsets[c+1]).  Rows whose offsets run
 * backwards or past num_refs / num_tokens, or whose id is
 * CLAIM_RESERVED_ID, are malformed: never accepted, UNKNOWN at check.  Rows
 * after a backwards row may share entries with earlier rows: each
 * well-formed row is still a claim of its own (claim_offload then stores
 * each claim's footprint separately, one extra wait for the stream). 
 * Claim ids are stable and distinct from request ids (Table 5).
 *
 * predicate_tokens gives each claim's materialization predicate
 * leading_prefix_at_least(k) (section 1 running example, k = 448; Table 5
 * fixed predicate): the claim is materialized when the blocks holding its
 * first k tokens (ceil(k / block_size) leading block-table positions) are
 * restored intact.  It is read by claim_offload only and fixed at
 * acceptance; NULL, or k >= the claim's tokens, means the whole claim.  A
 * failed block past the predicate does not fail the claim (it sets
 * CLAIM_R_BEYOND_PREDICATE); ambiguity anywhere still gives UNKNOWN. */
typedef struct claim_batch {
  uint32_t num_claims;
  uint32_t reserved; /* must be 0 */
  uint64_t num_refs; /* entries in block_ids, < 2^32 */
  uint64_t num_tokens;
  const uint64_t* claim_ids;     /* [num_claims] */
  const uint32_t* block_offsets; /* [num_claims + 1] */
  const uint32_t* block_ids;     /* [num_refs] */
  const uint64_t* token_offsets; /* [num_claims + 1] */
  const uint32_t* tokens;        /* [num_tokens] */
  const uint64_t* predicate_tokens; /* [num_claims] or NULL: see above */
} claim_batch;

/* Faults applied by claim_restore (host memory, read before it returns).
 * flip f XORs canonical bit flip_bits[f] (bit 0 = least significant bit of
 * canonical byte 0) of block flip_blocks[f]; a bit flipped twice is
 * restored.  load_failed_blocks are reported load failures (section 7 path
 * B, the controlled CPU->GPU load failure F0): each fails, at that block,
 * every claim whose offload recorded the block before this restore, and
 * nothing clears it for them.  A later offload of the block (a recompute
 * stored under another claim) is that claim's own record: it does not
 * restore the earlier claims (Table 9, fallback-recompute row), and the
 * earlier failure is not the later claim's failure. */
typedef struct claim_fault_spec {
  uint32_t num_flips;
  uint32_t num_load_failed;
  const uint32_t* flip_blocks; /* [num_flips], each < num_blocks */
  const uint64_t* flip_bits;   /* [num_flips], each < 8 * block bytes */
  const uint32_t* load_failed_blocks; /* [num_load_failed], each < num_blocks */
} claim_fault_spec;

/* One claim's outcome (64 bytes). */
typedef struct claim_outcome {
  uint64_t claim_id;
  uint32_t code;                /* CLAIM_UNKNOWN / _MATERIALIZED / _RESTORE_FAILED_FAIL_CLOSED */
  uint32_t first_failing_block; /* position j* in the claim, CLAIM_NONE if none */
  uint32_t phys_block;          /* block-table entry at j* (CLAIM_NONE if j* >= blocks) */
  uint32_t num_blocks;          /* block-table entries presented (0 if malformed) */
  uint32_t reasons;             /* OR of CLAIM_R_* found anywhere in the claim */
  uint32_t intact_blocks;       /* leading positions with no problem at all (<= num_blocks) */
  uint64_t expected_digest;     /* the claim's own offload digest at j* (failures only, else 0) */
  uint64_t observed_digest;     /* restored digest at j* (failures only, else 0) */
  uint64_t chain_hash;          /* h_{nt-1} of the presented tokens (S if none) */
  uint64_t chain_hash_at_fail;  /* h_{j*} if j* < nt, else 0 */
} claim_outcome;

/* One lifecycle event (40 bytes).  aux by kind: ACCEPTED = chain hash;
 * OFFLOADED = blocks; RESTORE_REQUIRED = accepted blocks; RESTORED = chain
 * hash; RESTORATION_FAILED = observed digest at the failing block;
 * ACTIVE_REQUEST_REFUSED = blocking claim id (the claim itself);
 * OUTCOME_UNKNOWN = reason bits. */
typedef struct claim_event {
  uint64_t seq;         /* position in the pool's global event order */
  uint64_t claim_id;
  uint64_t aux;
  uint32_t kind;        /* CLAIM_EV_* */
  uint32_t block_index; /* j, CLAIM_NONE if none */
  uint32_t phys_block;  /* CLAIM_NONE if none */
  uint32_t reserved;
} claim_event;

/* Result of a reuse lookup for one request row (40 bytes). */
#define CLAIM_LOOKUP_UNKNOWN 0 /* malformed row, or the lookup reached an ambiguous identity */
#define CLAIM_LOOKUP_HIT 1     /* every token block of the request hit */
#define CLAIM_LOOKUP_PARTIAL 2 /* a leading run of token blocks hit, not all */
#define CLAIM_LOOKUP_MISS 3    /* no token block hit (or the request has no tokens) */

typedef struct claim_lookup_result {
  uint64_t request_id;        /* claim_ids[c] of the request row */
  uint64_t hit_tokens;        /* min(hit_blocks * block_size, request tokens) */
  uint64_t chain_hash_at_hit; /* h_{hit_blocks-1}; the pool seed S when hit_blocks = 0 */
  uint32_t status;            /* CLAIM_LOOKUP_* */
  uint32_t hit_blocks;        /* leading token blocks whose identity is registered and unambiguous */
  uint32_t last_block;        /* physical block registered for h_{hit_blocks-1}; CLAIM_NONE if none */
  uint32_t reserved;
} claim_lookup_result;

/* Stage times of the claim_check calls queued since the last
 * claim_timing_read, measured with hipEvents on the pool's stream.  With
 * CLAIM_POOL_TIMING only digest_ms is filled (two events per check around
 * the gather + digest kernel); with CLAIM_POOL_STAGE_TIMING as well, every
 * field. */
typedef struct claim_timing {
  uint32_t calls;          /* checks measured */
  uint32_t last_unique;    /* unique blocks digested by the last check */
  double total_ms;         /* sum over calls: whole check (stage timing) */
  double digest_ms;        /* sum over calls: the gather + digest kernel */
  double select_ms;        /* sum over calls: unique-block selection (stage timing) */
  double finalize_ms;      /* sum over calls: per-block digest combine (stage timing) */
  double claims_ms;        /* sum over calls: chain, compare, min-reduction, outcomes (stage timing) */
  double events_ms;        /* sum over calls: event scan and append (stage timing) */
} claim_timing;

/* Create a pool over caller-owned KV memory (section 7: the connector's
 * accepted-claim state; Table 5: fixed cache identity = seed + geometry).
 * Allocates the pool's device state: per block the latest offload digest,
 * the restored digest and latest reported-failure generation (16 bytes),
 * whether some claim recorded it, and the identity of its latest
 * registration; the claim registry (ids, state, token count, chain hash,
 * footprint, offload generation; per position the accepted identity and the
 * claim's own offload digest: 20 bytes per footprint entry); the
 * cache-identity table (32 bytes per entry: the entry and where its first
 * registrant keeps its accepted identities; next_pow2(2 * max_footprint)
 * entries), the event log and scratch.  Returns EINVAL for a bad
 * description, ENOMEM / EHIP on allocation failure. */
int claim_pool_create(const claim_pool_desc* desc, claim_pool** out);

/* Wait for the pool's stream, then free everything the pool owns (not the
 * KV memory): the end of the connector state of section 7, after which no
 * claim of the pool can be restored or checked.  NULL is accepted. */
int claim_pool_destroy(claim_pool* pool);

/* Accept and offload a batch (section 1: accept, materialized, offloaded;
 * section 5 storage_restorability: the claim is accepted before offload).
 * The whole batch is refused with EDUP if a non-reserved id occurs twice or
 * is already registered (Table 2: duplicate ownership fails closed); nothing
 * changes then.  Otherwise each well-formed claim is registered (event
 * ACCEPTED) with its own offload record: the digest of every in-range
 * block it references, taken by this call (section 5 storage_restorability:
 * store and load name the same claim), so no later offload of a shared
 * block by another claim changes what the claim is checked against.  A
 * claim whose footprint is non-empty, fully present and equal in length to
 * ceil(tokens/block_size) becomes OFFLOADED (event OFFLOADED).  Each
 * claim's accepted identity h_j (its chain hash after token block j) is
 * kept for every position with both a block and tokens.  For every
 * OFFLOADED claim, (h_j -> block j) is registered in the cache-identity
 * table (section 5 cache identity; Table 5 joinable block hashes): a
 * registration equal to an existing one is stored once; the same identity
 * registered to a different block is duplicate ownership and makes the
 * identity ambiguous (Table 2).  A block holds the identity of its latest
 * registration (in call, then batch, then position order); identities it
 * held before are stale and no longer hit in claim_lookup.  Entries are
 * never removed.  With staging != NULL the canonical bytes of every such
 * block are also written to staging (device memory or host memory from
 * hipHostMalloc, 16-byte aligned, else EINVAL), one block after another in
 * ascending block-id order, as the offload tier of section 7 paths A and B.
 * Staged offloads into the same staging buffer accumulate: each appends its
 * blocks after those the buffer already holds, and a block's staged copy is
 * its latest staged offload's.  staging_bytes must cover the blocks already
 * there and this offload's (else ENOSPC).  A staged offload into another
 * buffer starts a new generation, as does claim_staging_reset: the blocks
 * staged before are no longer restored from staging.  An offload without
 * staging drops the staged copies of its blocks (they are no longer the
 * bytes of the block's latest offload).  A block with no staged copy is used
 * as the pool holds it (a claim whose bytes are gone fails closed on its
 * digest compare), although lookups may still hit its identity.  Stores
 * are not deduplicated across calls: a block staged again takes a new slot.
 * Waits twice
 * for the stream to read the acceptance verdict (three times when a block
 * row runs backwards).  ENOSPC if the registry, footprint store or event
 * log could overflow; the footprint store takes num_refs entries, or, when
 * rows share entries, the sum of the well-formed rows' lengths.
 */
int claim_offload(claim_pool* pool, const claim_batch* batch, void* staging,
                  uint64_t staging_bytes);

/* Restore (section 7 path A steps 4-5, path B steps 3-5).  If staging is
 * not NULL it must be the buffer of the pool's current staging generation
 * (staging_bytes covering every slot staged to it, else EINVAL): every
 * block with a staged copy that a well-formed claim of the batch references
 * is copied back into the pool from that copy.  Then the faults are applied (faults may be NULL).  Then each
 * well-formed, registered and OFFLOADED claim of the batch moves to
 * RESTORE_REQUIRED (event RESTORE_REQUIRED).  EINVAL for an out-of-range
 * fault or a staging pointer that is not 16-byte aligned. */
int claim_restore(claim_pool* pool, const claim_batch* batch, const void* staging,
                  uint64_t staging_bytes, const claim_fault_spec* faults);

/* Start a new staging generation (section 7 paths A and B: the offload
 * tier): no block keeps a staged copy, and the next staged offload writes
 * from the start of its buffer, whichever buffer it is.  For a caller that
 * reuses one staging buffer for unrelated offloads.  Queued on the pool's
 * stream; EINVAL for a NULL pool. */
int claim_staging_reset(claim_pool* pool);

/* Check (section 7 path A step 5, path B steps 5-7, path C): digest every
 * in-range block with an offload record that the well-formed claims
 * reference, and judge each claim's blocks against its own offload record:
 * a load failure reported after its offload, or a restored digest that
 * differs from its own offload digest, is a restoration failure at that
 * position; an entry that is not the accepted one holds no record of the
 * claim (CLAIM_R_NO_OFFLOAD_RECORD, with CLAIM_R_FOOTPRINT_MISMATCH).
 * Chain each claim's tokens and decide its outcome.
 * The cache identity is compared position by position: a token block whose
 * h_j differs from the accepted one, or the block where the token counts
 * part (min(tokens, accepted tokens) / block_size), is an ambiguity at that
 * position (CLAIM_R_TOKEN_MISMATCH); a different whole-claim chain hash is
 * also a claim-level ambiguity.  The smallest key (class << 32 | position)
 * over the claim's problems wins,
 * class 0 = ambiguity -> UNKNOWN, class 1 = load failure or digest mismatch
 * -> RESTORE_FAILED_FAIL_CLOSED, none -> MATERIALIZED.  Appends, in batch
 * order, RESTORED, or RESTORATION_FAILED then ACTIVE_REQUEST_REFUSED (the
 * claim is its own blocking id), or OUTCOME_UNKNOWN.  The registry is not
 * changed.  ENOSPC if the event log could overflow. */
int claim_check(claim_pool* pool, const claim_batch* batch);

/* claim_check for callers that cannot allocate memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  It does
 * the same work with the same kernels and the same results, but allocates
 * nothing: its per-claim scratch (event counts, pending events, event-scan
 * tile sums; 36 bytes per claim) lives in one fixed device array per GPU of
 * about 9.4 MB, which the library holds until the process ends, and the
 * outcomes go to `out` (device memory, capacity out_cap records), not to
 * the pool.  Events are appended to the pool's log as by claim_check and
 * read with outcomes_read, which then reports no outcomes (they are in
 * `out`, complete once the pool's stream reaches this call; the call does
 * not wait).  Batches of more than CLAIM_STATIC_MAX_CLAIMS claims return
 * CLAIM_ELIMIT; out_cap < num_claims or a log that could overflow return
 * CLAIM_ENOSPC; a NULL out with claims returns CLAIM_EINVAL; nothing is
 * queued then.  Every call on one GPU, from any pool, shares that GPU's
 * array, and each call overwrites what the previous one left there: calls
 * that overlap on one GPU (pools on different streams, or host threads)
 * race and must be serialized by the caller.  Nothing in the array needs to
 * start at zero: each call writes every entry it reads.  On a pool created
 * without timing flags the call only queues kernels, so it can be captured
 * into a HIP graph; each replay checks the batch again and appends its
 * events (all or none: see outcomes_read), and the caller reads or resets
 * the log between replays as between calls. */
#define CLAIM_STATIC_MAX_CLAIMS 262144u
int claim_check_static(claim_pool* pool, const claim_batch* batch, claim_outcome* out,
                       uint32_t out_cap);

/* Reuse lookup (section 7 paths A and B, order 3: the lookup reports how
 * many of the request's tokens hit the offloaded claim footprint, hit=448
 * in the running example).  For each request row c of the batch (its id,
 * token_offsets and tokens; block rows are not read and may be NULL): the
 * chain h_0 .. h_{nt-1} of its tokens, and hit_blocks = the number of
 * leading token blocks whose identity is registered, unambiguous and still
 * held by its block (a block registered since under another identity no
 * longer holds this prefix: the stale identity stops the lookup as an
 * absent one does).  The lookup stops at the first block that is not; if
 * that identity is
 * registered but ambiguous (duplicate ownership), the status is
 * CLAIM_LOOKUP_UNKNOWN rather than a shorter hit (Table 2: duplicate owners
 * fail closed), as it is for a malformed row (reserved id, token offsets
 * that run backwards or past num_tokens).  The registry and event log are
 * not changed.  out is device memory with room for out_cap records; it is
 * written in stream order on the pool's stream and is complete once the
 * stream reaches this call (the call does not wait).  ENOSPC if out_cap <
 * num_claims; EINVAL for a NULL out with requests, or a bad batch. */
int claim_lookup(claim_pool* pool, const claim_batch* requests, claim_lookup_result* out,
                 uint32_t out_cap);

/* Wait for the pool's stream and return the number of registered
 * identities and how many of them are ambiguous (registered to two or more
 * different blocks).  Either pointer may be NULL. */
int claim_identity_stats(claim_pool* pool, uint64_t* entries, uint64_t* ambiguous);

/* The section 7 event stream and claim outcomes, read out (paths A and B:
 * the ordered events E0 .. E13 and the claim-scoped outcome; section 1
 * running example, the accepted event sequence).
 * Wait for the pool's stream and copy to the host the outcomes of the last
 * claim_check (into out, capacity out_cap; *num_out = their count) and the
 * events appended since the previous outcomes_read (into events, capacity
 * ev_cap; *num_events = their count), which are then dropped from the log
 * (sequence numbers keep counting).  A NULL out or events skips that part
 * (events are then kept).  ENOSPC, with nothing copied or dropped, if a
 * capacity is too small.  Every call checks on the host that its events
 * fit the log before it queues work; the device also appends each call's
 * events all or none, so work the host did not bound (a captured
 * claim_check_static replayed from a graph) can never write past the log:
 * a call whose events did not fit appends none and marks the log, and the
 * next outcomes_read copies what the log holds, clears the mark when it
 * reads the events, and returns ENOSPC. */
int outcomes_read(claim_pool* pool, claim_outcome* out, uint32_t out_cap, uint32_t* num_out,
                  claim_event* events, uint64_t ev_cap, uint64_t* num_events);

/* The digest grid of a pool.  A digest launch runs slots resident
 * workgroups of 4 waves; each wave reads one piece (64 lanes x
 * words_per_lane 8-byte words) of one plane's chunk of each block it
 * visits, a workgroup 4 consecutive pieces (a piece group), and the launch
 * reads pga piece groups at a time with groups workgroups on each. */
typedef struct claim_grid_info {
  uint32_t words_per_lane;  /* 8-byte words per lane in one piece */
  uint32_t segments;        /* pieces per plane chunk */
  uint32_t piece_groups;    /* ceil(planes x segments / 4) */
  uint32_t slots;           /* workgroups resident at once (per CU x CUs) */
  uint32_t pga;             /* a launch over `refs` entries: piece groups read at a time */
  uint32_t groups;          /* ... and workgroups on each */
} claim_grid_info;

/* Report the digest grid (claim_grid_info) that a launch over a batch of
 * `refs` block-table entries takes (the piece groups read at a time follow
 * from an upper bound on the launch's unique blocks, min(refs,
 * num_blocks)).  Does not wait or queue work.  EINVAL for a NULL pool or
 * out. */
int claim_digest_grid(const claim_pool* pool, uint64_t refs, claim_grid_info* out);

/* Wait for the pool's stream and return the summed stage times of the
 * checks queued since the previous call (EINVAL unless the pool was created
 * with CLAIM_POOL_TIMING or CLAIM_POOL_STAGE_TIMING). */
int claim_timing_read(claim_pool* pool, claim_timing* out);

/* Wait for the pool's stream and copy the per-block state of blocks
 * [first, first + count) to the host: the digest recorded by the block's
 * latest offload (each claim is checked against its own record, which the
 * outcome reports as expected_digest), restored digests D_res (as of the
 * last check that digested the block), whether some claim recorded the
 * block, and whether a load failure of it has ever been reported (one byte
 * each, 0 or 1).  Any output pointer may be NULL.  EINVAL if the range
 * exceeds the pool.  This is the block-level evidence behind a claim
 * outcome (section 7 path B step 5: affected-block evidence). */
int claim_block_state_read(claim_pool* pool, uint32_t first, uint32_t count, uint64_t* d_off,
                           uint64_t* d_res, uint8_t* valid_off, uint8_t* load_failed);

/* Text for a status code (static storage).  Status codes report API misuse
 * and resource limits only; claim problems are outcomes, never statuses
 * (Table 2: ambiguity yields no claim outcome rather than an error). */
const char* claim_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* CLAIMKV_H */
