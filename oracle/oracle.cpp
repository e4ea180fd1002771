/*
 * oracle.cpp -- reference oracle for claim-scoped KV materialization checking.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke entry point and
 * the benchmark's CPU-baseline leg may load this library.  The product path
 * (the HIP library and its Python binding) never links, loads or calls it,
 * and it shares no source, header, table or helper with that path.
 *
 * It is deliberately plain: single-threaded loops that follow the
 * definitions one statement at a time, with no blocking, fusion or
 * reordering, so that a reader can check it against the definitions below
 * by eye.  Speed is not a goal.
 *
 * What is computed, and where it comes from:
 *
 *  - Claim semantics (the paper, "Fail-Closed Lowering of Resident KV Claims
 *    onto LLM Serving Runtimes"):
 *      * a claim is an accepted future-reuse responsibility with a stable id,
 *        a footprint and a predicate (section 1, Table 1 claim_identity,
 *        explicit_acceptance, materialization_predicate);
 *      * lifecycle order accept -> offloaded -> restore-required -> restored,
 *        or -> restoration_failed -> active_request_refused with the claim in
 *        blocking_claim_ids (section 1 running example; section 7 event list
 *        E0..E14 and witness paths A and B);
 *      * only failures of the claim's own blocks count (section 7 path C,
 *        Table 9 last row);
 *      * offload records are the claim's own: at acceptance a claim keeps the
 *        digest of each of its blocks, and its check compares against those,
 *        so another claim's later offload of a shared block neither satisfies
 *        nor changes it (section 5 storage_restorability row: store and load
 *        name the same claim; a recompute must not be relabelled as
 *        restoration; Table 9 wrong-claim and fallback-recompute rows);
 *      * a reported load failure fails every claim that recorded the block
 *        before the report, and nothing clears it for them: a later offload
 *        of the block (a recompute stored by another claim) is that claim's
 *        own record (Table 9, fallback-recompute row);
 *      * ambiguity yields no claim outcome (Table 2, last rule; Table 5, last
 *        row): missing registry, unstable ids, cache-identity mismatch,
 *        partial streams and duplicate ownership all give UNKNOWN here.
 *  - Arithmetic (the paper fixes none: it never defines a digest or hash; this
 *    checker's definitions, recorded with the rest of the design):
 *      * mix64 / splitmix64: the SplitMix64 generator of Steele, Lea and Flood
 *        (OOPSLA 2014), written here from its published description;
 *      * KV word keys k_i = splitmix64(S, i) | 1 and the block digest
 *        D = sum_i w_i * k_i mod 2^64 over little-endian 64-bit words of the
 *        block's canonical bytes;
 *      * token keys t_m = splitmix64(~S, m) | 1, the per-block token
 *        multilinear M_j = sum_m tok * t_m, and the chain
 *        h_{-1} = S, h_j = splitmix64(h_{j-1} xor M_j).
 *  - Cache identity (section 5 cache_identity; Table 5 fixed cache identity
 *    and joinable block hashes; section 7 reuse lookup E1 reporting a hit):
 *    h_j names the token prefix held by a claim's j-th block.  Offload
 *    registers (h_j -> physical block) for every offloaded claim; equal
 *    registrations are stored once, and one identity registered to two
 *    different blocks is duplicate ownership, which makes the identity
 *    ambiguous.  A block holds the identity of its latest registration; an
 *    identity whose block was since registered under another identity is
 *    stale (the block no longer holds that prefix).  A lookup reports the
 *    longest leading run of a request's token blocks whose identities are
 *    registered, unambiguous and still held by their block.  The check
 *    compares each h_j of the presented tokens with the one accepted for
 *    that position.
 *
 * Parity pins (checked by the CPU tests): the published SplitMix64 outputs
 * for seed 0; D(0) = 0, D(e_i) = k_i, additivity, the exact single-bit-flip
 * delta +-2^beta * k_i; exhaustive single flips on a small block; head-shard
 * digests that add up to the block digest over a partition of the heads and
 * equal the digest of the block with the other heads zeroed; four
 * token blocks whose chain h_0 .. h_3 is the published SplitMix64 stream
 * for seed 0; shared token prefixes give equal chain hashes; outcome
 * enumeration over every ok/failed/missing assignment of short claims, with
 * every predicate length; memcmp brute force of the failing set on the tiny
 * pool; a claim ledger (each claim's own stored copy of its blocks, failures
 * reported after it, compared by memcmp) over random lifecycles with several
 * offloads, block rewrites and recomputes; brute-force walks over
 * token-prefix tuples, with the prefix each block holds, for the identity
 * table and the lookup; event payloads against values computed without the
 * lifecycle (counts, reason bits, the exact single-flip digest delta); the
 * paper's event-order templates and its 448-token and 17-token examples.
 */

#include <cstdint>
#include <cstring>
#include <unordered_map>
#include <vector>

namespace {

/* ---------------------------------------------------------------- hashing */

const uint64_t kGamma = 0x9E3779B97F4A7C15ull; /* SplitMix64 increment */

/* SplitMix64 output (finaliser) function. */
uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* One SplitMix64 step from state x: advance by gamma, then finalise. */
uint64_t splitmix64(uint64_t x) { return mix64(x + kGamma); }

/* The (i+1)-th output of the SplitMix64 stream whose state starts at s. */
uint64_t splitmix64_at(uint64_t s, uint64_t i) { return mix64(s + (i + 1) * kGamma); }

uint64_t kv_key(uint64_t seed, uint64_t i) { return splitmix64_at(seed, i) | 1ull; }

uint64_t token_key(uint64_t seed, uint64_t m) { return splitmix64_at(~seed, m) | 1ull; }

/* Little-endian 64-bit word from 8 bytes, one byte at a time. */
uint64_t le_word(const uint8_t* p) {
  uint64_t w = 0;
  for (int k = 0; k < 8; ++k) w |= (uint64_t)p[k] << (8 * k);
  return w;
}

/* Block digest over canonical bytes: sum over words of w_i * k_i mod 2^64. */
uint64_t block_digest(const uint8_t* canon, uint64_t nbytes, uint64_t seed) {
  uint64_t d = 0;
  for (uint64_t i = 0; i < nbytes / 8; ++i) d += le_word(canon + 8 * i) * kv_key(seed, i);
  return d;
}

/* Digest of a head shard of a block (a pool that holds KV heads
 * [first_head, first_head + heads) of blocks whose full width is heads_total
 * heads, as under tensor parallelism by KV head).  The full block's canonical
 * bytes are its planes' chunks in order, each chunk [token][head][row_bytes];
 * the shard's own canonical bytes are the same with only its heads.  Each
 * shard word keeps the key of its position in the full block, so this is the
 * full block's digest restricted to the shard's words, and the shards of a
 * block add up to its digest.  row_bytes (one head's bytes of one token) is a
 * multiple of 8. */
uint64_t shard_digest(const uint8_t* canon, uint32_t planes, uint32_t block_size, uint32_t heads,
                      uint32_t row_bytes, uint32_t heads_total, uint32_t first_head,
                      uint64_t seed) {
  const uint64_t row_words = row_bytes / 8;
  uint64_t d = 0;
  for (uint64_t p = 0; p < planes; ++p)
    for (uint64_t t = 0; t < block_size; ++t)
      for (uint64_t h = 0; h < heads; ++h)
        for (uint64_t w = 0; w < row_words; ++w) {
          const uint64_t local_word = ((p * block_size + t) * heads + h) * row_words + w;
          const uint64_t full_word =
              ((p * block_size + t) * heads_total + first_head + h) * row_words + w;
          d += le_word(canon + 8 * local_word) * kv_key(seed, full_word);
        }
  return d;
}

/* Token multilinear of one token block: sum over present tokens of tok * t_m. */
uint64_t token_multilinear(const uint32_t* tok, uint64_t n, uint64_t seed) {
  uint64_t m_sum = 0;
  for (uint64_t m = 0; m < n; ++m) m_sum += (uint64_t)tok[m] * token_key(seed, m);
  return m_sum;
}

uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

/* Chain over a claim's tokens: h_{-1} = S, h_j = splitmix64(h_{j-1} ^ M_j).
 * Writes h_0 .. h_{nt-1} (nt = ceil(ntok / bs)) and returns h_{nt-1}, or S
 * when there are no tokens. */
uint64_t chain(const uint32_t* tok, uint64_t ntok, uint32_t bs, uint64_t seed,
               std::vector<uint64_t>* h_out) {
  uint64_t h = seed;
  uint64_t nt = ceil_div(ntok, bs);
  if (h_out) h_out->assign(nt, 0);
  for (uint64_t j = 0; j < nt; ++j) {
    uint64_t first = j * bs;
    uint64_t count = ntok - first < bs ? ntok - first : bs;
    uint64_t m_sum = token_multilinear(tok + first, count, seed);
    h = splitmix64(h ^ m_sum);
    if (h_out) (*h_out)[j] = h;
  }
  return h;
}

/* ------------------------------------------------------------ vocabulary */

const uint32_t kNone = 0xFFFFFFFFu;
const uint64_t kReservedId = 0xFFFFFFFFFFFFFFFFull;

enum { ST_ACCEPTED = 1, ST_OFFLOADED = 2, ST_RESTORE_REQUIRED = 4 };

enum {
  OUT_UNKNOWN = 0,
  OUT_MATERIALIZED = 1,
  OUT_RESTORE_FAILED_FAIL_CLOSED = 2,
};

enum {
  EV_ACCEPTED = 1,
  EV_OFFLOADED = 2,
  EV_RESTORE_REQUIRED = 3,
  EV_RESTORED = 4,
  EV_RESTORATION_FAILED = 5,
  EV_ACTIVE_REQUEST_REFUSED = 6,
  EV_OUTCOME_UNKNOWN = 7,
};

enum {
  R_NOT_ACCEPTED = 0x001,
  R_NOT_OFFLOADED = 0x002,
  R_NO_RESTORE = 0x004,
  R_TOKEN_MISMATCH = 0x008,
  R_FOOTPRINT_MISMATCH = 0x010,
  R_MISSING_ENTRY = 0x020,
  R_NO_OFFLOAD_RECORD = 0x040,
  R_SHAPE_MISMATCH = 0x080,
  R_EMPTY = 0x100,
  R_MALFORMED = 0x200,
  R_LOAD_FAILED = 0x400,
  R_DIGEST_MISMATCH = 0x800,
  R_BEYOND_PREDICATE = 0x1000,
};

enum { LK_UNKNOWN = 0, LK_HIT = 1, LK_PARTIAL = 2, LK_MISS = 3 };

enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_EDUP = -5 };

}  // namespace

extern "C" {

/* Records handed back to the tests (the oracle's own layout). */
typedef struct orc_outcome {
  uint64_t claim_id;
  uint32_t code;
  uint32_t first_failing_block;
  uint32_t phys_block;
  uint32_t num_blocks;
  uint32_t reasons;
  uint32_t intact_blocks;
  uint64_t expected_digest;
  uint64_t observed_digest;
  uint64_t chain_hash;
  uint64_t chain_hash_at_fail;
} orc_outcome;

typedef struct orc_lookup {
  uint64_t request_id;
  uint64_t hit_tokens;
  uint64_t chain_hash_at_hit;
  uint32_t status;
  uint32_t hit_blocks;
  uint32_t last_block;
  uint32_t pad;
} orc_lookup_result;

typedef struct orc_event {
  uint64_t seq;
  uint64_t claim_id;
  uint64_t aux;
  uint32_t kind;
  uint32_t block_index;
  uint32_t phys_block;
  uint32_t pad;
} orc_event;

}  // extern "C"

namespace {

struct Claim {
  uint32_t state;
  std::vector<uint32_t> footprint;
  uint64_t n_tokens;
  uint64_t chain_hash;
  uint32_t pred_blocks; /* leading positions the predicate covers */
  std::vector<uint64_t> identity; /* accepted h_j for j < min(blocks, token blocks) */
  /* the claim's own offload record: the digest of the block at each
   * in-range footprint position when the claim was offloaded (0 where the
   * entry is missing), and the generation of that offload */
  std::vector<uint64_t> digest;
  uint64_t generation;
};

/* One registered cache identity: the physical block that holds it, and
 * whether a second, different block was also registered for it. */
struct Identity {
  uint32_t block;
  bool ambiguous;
};

/* Pool state.  Every offload and every restore call takes the next
 * generation, so generations order the lifecycle calls.  Per block:
 * d_off = the digest recorded by the block's latest offload, valid_off =
 * some claim holds an offload record of it, d_res = its digest at the last
 * check that re-digested it, fail_gen = the generation of its latest
 * reported load failure (0 = none), holder = the identity of its latest
 * registration (meaningful once the block has been registered). */
struct Pool {
  uint32_t num_blocks;
  uint32_t block_size;
  uint64_t seed;
  uint64_t generation;
  std::vector<uint64_t> d_off, d_res, fail_gen, holder;
  std::vector<uint8_t> valid_off;
  std::unordered_map<uint64_t, Claim> registry;
  std::unordered_map<uint64_t, Identity> identities;
  std::vector<orc_event> log;
  uint64_t next_seq;
};

/* A read-only view of one claim batch (compressed rows). */
struct Batch {
  uint32_t num_claims;
  uint64_t num_refs;
  uint64_t num_tokens;
  const uint64_t* ids;
  const uint32_t* blk_off;
  const uint32_t* blk_ids;
  const uint64_t* tok_off;
  const uint32_t* tokens;
};

/* A claim row is malformed when its offsets run backwards or past the end of
 * the arrays, or when it uses the reserved id.  Malformed rows are never
 * accepted and check as UNKNOWN. */
bool malformed(const Batch& bt, uint32_t c) {
  if (bt.ids[c] == kReservedId) return true;
  if (bt.blk_off[c] > bt.blk_off[c + 1] || bt.blk_off[c + 1] > bt.num_refs) return true;
  if (bt.tok_off[c] > bt.tok_off[c + 1] || bt.tok_off[c + 1] > bt.num_tokens) return true;
  return false;
}

void append_event(Pool* p, uint64_t claim_id, uint32_t kind, uint32_t j, uint32_t phys,
                  uint64_t aux) {
  orc_event e;
  e.seq = p->next_seq++;
  e.claim_id = claim_id;
  e.aux = aux;
  e.kind = kind;
  e.block_index = j;
  e.phys_block = phys;
  e.pad = 0;
  p->log.push_back(e);
}

}  // namespace

extern "C" {

/* -------------------------------------------------------- pure functions */

uint64_t orc_mix64(uint64_t z) { return mix64(z); }
uint64_t orc_splitmix64(uint64_t x) { return splitmix64(x); }
uint64_t orc_splitmix64_at(uint64_t s, uint64_t i) { return splitmix64_at(s, i); }
uint64_t orc_kv_key(uint64_t seed, uint64_t i) { return kv_key(seed, i); }
uint64_t orc_token_key(uint64_t seed, uint64_t m) { return token_key(seed, m); }

uint64_t orc_block_digest(const uint8_t* canon, uint64_t nbytes, uint64_t seed) {
  return block_digest(canon, nbytes, seed);
}

uint64_t orc_shard_digest(const uint8_t* canon, uint32_t planes, uint32_t block_size,
                          uint32_t heads, uint32_t row_bytes, uint32_t heads_total,
                          uint32_t first_head, uint64_t seed) {
  return shard_digest(canon, planes, block_size, heads, row_bytes, heads_total, first_head, seed);
}

uint64_t orc_token_multilinear(const uint32_t* tok, uint64_t n, uint64_t seed) {
  return token_multilinear(tok, n, seed);
}

/* Chain hashes h_0 .. h_{nt-1} of one claim's tokens; returns h_{nt-1} (S if
 * there are no tokens).  h_out may be NULL. */
uint64_t orc_chain(const uint32_t* tok, uint64_t ntok, uint32_t bs, uint64_t seed,
                   uint64_t* h_out) {
  std::vector<uint64_t> h;
  uint64_t last = chain(tok, ntok, bs, seed, &h);
  if (h_out)
    for (uint64_t j = 0; j < h.size(); ++j) h_out[j] = h[j];
  return last;
}

/* Canonical bytes of block b: the concatenation over planes p = 0..P-1 of
 * the chunk of plane p, where the pool is laid out [plane][block][chunk]. */
int orc_canonical_block(const uint8_t* pool, uint32_t planes, uint32_t num_blocks,
                        uint64_t chunk_bytes, uint32_t b, uint8_t* out) {
  if (b >= num_blocks) return ORC_EINVAL;
  for (uint32_t p = 0; p < planes; ++p) {
    const uint8_t* src = pool + ((uint64_t)p * num_blocks + b) * chunk_bytes;
    for (uint64_t q = 0; q < chunk_bytes; ++q) out[(uint64_t)p * chunk_bytes + q] = src[q];
  }
  return ORC_OK;
}

/* The block digest of every block of a host pool laid out
 * [plane][block][chunk]: block b's canonical bytes (as orc_canonical_block
 * forms them) digested with block_digest, one block after another.  Only a
 * loop over the single-block definition, for pools with millions of
 * blocks. */
int orc_pool_digests(const uint8_t* pool, uint32_t planes, uint32_t num_blocks,
                     uint64_t chunk_bytes, uint64_t seed, uint64_t* out) {
  if ((planes * chunk_bytes) % 8) return ORC_EINVAL;
  std::vector<uint8_t> canon(planes * chunk_bytes);
  for (uint32_t b = 0; b < num_blocks; ++b) {
    orc_canonical_block(pool, planes, num_blocks, chunk_bytes, b, canon.data());
    out[b] = block_digest(canon.data(), canon.size(), seed);
  }
  return ORC_OK;
}

/* Flip canonical bit `bit` of block b in place (bit 0 = least significant
 * bit of canonical byte 0). */
int orc_apply_flip(uint8_t* pool, uint32_t planes, uint32_t num_blocks, uint64_t chunk_bytes,
                   uint32_t b, uint64_t bit) {
  if (b >= num_blocks || bit >= 8 * chunk_bytes * planes) return ORC_EINVAL;
  uint64_t byte = bit / 8;
  uint64_t p = byte / chunk_bytes;
  uint64_t q = byte % chunk_bytes;
  pool[(p * num_blocks + b) * chunk_bytes + q] ^= (uint8_t)(1u << (bit % 8));
  return ORC_OK;
}

/* -------------------------------------------------------------- lifecycle */

void* orc_pool_new(uint32_t num_blocks, uint32_t block_size, uint64_t seed) {
  if (num_blocks == 0 || block_size == 0) return nullptr;
  Pool* p = new Pool();
  p->num_blocks = num_blocks;
  p->block_size = block_size;
  p->seed = seed;
  p->generation = 0;
  p->d_off.assign(num_blocks, 0);
  p->d_res.assign(num_blocks, 0);
  p->fail_gen.assign(num_blocks, 0);
  p->holder.assign(num_blocks, 0);
  p->valid_off.assign(num_blocks, 0);
  p->next_seq = 0;
  return p;
}

void orc_pool_free(void* handle) { delete static_cast<Pool*>(handle); }

/* Accept and offload a batch.  digest_now[b] is the digest of block b's
 * current bytes (only entries referenced by the batch are read).
 *
 * The whole batch is refused (ORC_EDUP, nothing changes, no event) if a
 * non-reserved id occurs twice in it or is already registered.  Otherwise
 * the call takes the next generation and, in batch order, each well-formed
 * claim is registered (ACCEPTED) with its own offload record (the digest of
 * every in-range block it references, and this generation), every such
 * block is marked as recorded, and a claim whose footprint is non-empty,
 * fully present and consistent with its token count is marked OFFLOADED
 * and registers its identities. */
int orc_offload(void* handle, uint32_t num_claims, uint64_t num_refs, uint64_t num_tokens,
                const uint64_t* ids, const uint32_t* blk_off, const uint32_t* blk_ids,
                const uint64_t* tok_off, const uint32_t* tokens, const uint64_t* predicate_tokens,
                const uint64_t* digest_now) {
  Pool* p = static_cast<Pool*>(handle);
  Batch bt = {num_claims, num_refs, num_tokens, ids, blk_off, blk_ids, tok_off, tokens};

  /* duplicate ownership refuses acceptance of the whole batch */
  std::unordered_map<uint64_t, int> seen;
  for (uint32_t c = 0; c < num_claims; ++c) {
    if (ids[c] == kReservedId) continue;
    if (p->registry.count(ids[c]) || seen.count(ids[c])) return ORC_EDUP;
    seen[ids[c]] = 1;
  }

  p->generation += 1;
  for (uint32_t c = 0; c < num_claims; ++c) {
    if (malformed(bt, c)) continue;
    uint32_t n = blk_off[c + 1] - blk_off[c];
    const uint32_t* fp = blk_ids + blk_off[c];
    uint64_t ntok = tok_off[c + 1] - tok_off[c];

    Claim cl;
    cl.state = ST_ACCEPTED;
    cl.footprint.assign(fp, fp + n);
    cl.generation = p->generation;
    cl.digest.assign(n, 0);
    for (uint32_t j = 0; j < n; ++j)
      if (fp[j] < p->num_blocks) cl.digest[j] = digest_now[fp[j]];
    cl.n_tokens = ntok;
    std::vector<uint64_t> h;
    cl.chain_hash = chain(tokens + tok_off[c], ntok, p->block_size, p->seed, &h);
    /* the accepted identity of every position that has both a block and tokens */
    uint64_t npos = n < h.size() ? n : h.size();
    cl.identity.assign(h.begin(), h.begin() + npos);
    /* leading_prefix_at_least(k): the blocks holding the first k tokens;
     * no predicate array means the whole claim */
    cl.pred_blocks = n;
    if (predicate_tokens && ceil_div(predicate_tokens[c], p->block_size) < n)
      cl.pred_blocks = (uint32_t)ceil_div(predicate_tokens[c], p->block_size);
    p->registry[ids[c]] = cl;
    append_event(p, ids[c], EV_ACCEPTED, kNone, kNone, cl.chain_hash);

    bool all_present = n > 0;
    for (uint32_t j = 0; j < n; ++j) {
      uint32_t b = fp[j];
      if (b >= p->num_blocks) {
        all_present = false;
        continue;
      }
      p->d_off[b] = digest_now[b];
      p->valid_off[b] = 1;
    }
    if (all_present && n == ceil_div(ntok, p->block_size)) {
      p->registry[ids[c]].state |= ST_OFFLOADED;
      append_event(p, ids[c], EV_OFFLOADED, kNone, kNone, n);
      /* register h_j -> block for each position of the offloaded claim: an
       * equal registration is stored once; a different block for the same
       * identity is duplicate ownership; the block now holds h_j */
      for (uint32_t j = 0; j < n; ++j) {
        auto it = p->identities.find(h[j]);
        if (it == p->identities.end()) {
          Identity idn;
          idn.block = fp[j];
          idn.ambiguous = false;
          p->identities[h[j]] = idn;
        } else if (it->second.block != fp[j]) {
          it->second.ambiguous = true;
        }
        p->holder[fp[j]] = h[j];
      }
    }
  }
  return ORC_OK;
}

/* Restore: take the next generation and record it as the latest reported
 * load failure of each listed block, then, in batch order, move every
 * well-formed, registered and offloaded claim to RESTORE_REQUIRED.  (Bit
 * flips act on bytes, see orc_apply_flip.) */
int orc_restore(void* handle, uint32_t num_claims, uint64_t num_refs, uint64_t num_tokens,
                const uint64_t* ids, const uint32_t* blk_off, const uint32_t* blk_ids,
                const uint64_t* tok_off, const uint32_t* tokens, uint32_t num_failed,
                const uint32_t* failed_blocks) {
  Pool* p = static_cast<Pool*>(handle);
  Batch bt = {num_claims, num_refs, num_tokens, ids, blk_off, blk_ids, tok_off, tokens};
  for (uint32_t f = 0; f < num_failed; ++f)
    if (failed_blocks[f] >= p->num_blocks) return ORC_EINVAL;
  p->generation += 1;
  for (uint32_t f = 0; f < num_failed; ++f) p->fail_gen[failed_blocks[f]] = p->generation;

  for (uint32_t c = 0; c < num_claims; ++c) {
    if (malformed(bt, c)) continue;
    auto it = p->registry.find(ids[c]);
    if (it == p->registry.end() || !(it->second.state & ST_OFFLOADED)) continue;
    it->second.state |= ST_RESTORE_REQUIRED;
    append_event(p, ids[c], EV_RESTORE_REQUIRED, kNone, kNone, it->second.footprint.size());
  }
  return ORC_OK;
}

/* Check: record restored digests, then decide each claim's outcome.
 *
 * The restored digest is refreshed for every in-range block with an offload
 * record that a well-formed row of the batch references.  Each position of
 * a registered claim is judged against the claim's own offload record of
 * the block at that position: a reported load failure later than the
 * claim's offload, or a restored digest different from the claim's own
 * offload digest, is a restoration failure there.  A position whose entry
 * differs from the accepted one (or lies past the accepted footprint) holds
 * no record of the claim.
 *
 * Every failure or ambiguity is a key (class << 32 | position); class 0 is
 * an ambiguity (no claim outcome), class 1 a restoration failure, and a
 * claim-level ambiguity sits at position NONE.  A failure beyond the
 * claim's predicate (the leading blocks its accepted
 * leading_prefix_at_least(k) covers, section 1 running example) is not a
 * key: it only sets the BEYOND_PREDICATE reason.  The smallest key decides:
 * none -> MATERIALIZED, class 0 -> UNKNOWN, class 1 ->
 * RESTORE_FAILED_FAIL_CLOSED.  Events are appended in batch order. */
int orc_check(void* handle, uint32_t num_claims, uint64_t num_refs, uint64_t num_tokens,
              const uint64_t* ids, const uint32_t* blk_off, const uint32_t* blk_ids,
              const uint64_t* tok_off, const uint32_t* tokens, const uint64_t* digest_now,
              orc_outcome* out) {
  Pool* p = static_cast<Pool*>(handle);
  Batch bt = {num_claims, num_refs, num_tokens, ids, blk_off, blk_ids, tok_off, tokens};

  /* restored digests of the recorded blocks the well-formed rows reference */
  for (uint32_t c = 0; c < num_claims; ++c) {
    if (malformed(bt, c)) continue;
    for (uint32_t i = blk_off[c]; i < blk_off[c + 1]; ++i) {
      uint32_t b = blk_ids[i];
      if (b < p->num_blocks && p->valid_off[b]) p->d_res[b] = digest_now[b];
    }
  }

  for (uint32_t c = 0; c < num_claims; ++c) {
    const uint64_t none_key = ((uint64_t)0 << 32) | kNone;
    uint64_t best = ~0ull; /* no key yet */
    uint32_t reasons = 0;
    uint32_t n = 0;
    uint64_t ntok = 0;
    const uint32_t* fp = nullptr;
    const uint32_t* tok = nullptr;

    if (malformed(bt, c)) {
      reasons |= R_MALFORMED;
      if (none_key < best) best = none_key;
    } else {
      n = blk_off[c + 1] - blk_off[c];
      fp = blk_ids + blk_off[c];
      ntok = tok_off[c + 1] - tok_off[c];
      tok = tokens + tok_off[c];
    }

    std::vector<uint64_t> h;
    uint64_t chain_hash = chain(tok, ntok, p->block_size, p->seed, &h);
    uint64_t nt = h.size();
    uint32_t pred = n;       /* predicate coverage: accepted value, else the whole claim */
    uint32_t intact = n;     /* first position with any problem, else n */
    const Claim* cl = nullptr;

    if (!(reasons & R_MALFORMED)) {
      auto it = p->registry.find(ids[c]);
      if (it == p->registry.end()) {
        reasons |= R_NOT_ACCEPTED;
        if (none_key < best) best = none_key;
      } else {
        cl = &it->second;
        pred = cl->pred_blocks < n ? cl->pred_blocks : n;
        if (!(cl->state & ST_OFFLOADED)) {
          reasons |= R_NOT_OFFLOADED;
          if (none_key < best) best = none_key;
        }
        if (!(cl->state & ST_RESTORE_REQUIRED)) {
          reasons |= R_NO_RESTORE;
          if (none_key < best) best = none_key;
        }
        /* cache identity position by position: a token block whose chain
         * hash differs from the accepted one, and the block where the token
         * counts part; the whole-claim hash remains a claim-level check */
        uint64_t npos = nt < cl->identity.size() ? nt : cl->identity.size();
        for (uint64_t j = 0; j < npos; ++j) {
          if (h[j] != cl->identity[j]) {
            reasons |= R_TOKEN_MISMATCH;
            uint64_t k = ((uint64_t)0 << 32) | j;
            if (k < best) best = k;
            if (j < intact) intact = (uint32_t)j;
          }
        }
        if (cl->n_tokens != ntok) {
          uint64_t q = (ntok < cl->n_tokens ? ntok : cl->n_tokens) / p->block_size;
          reasons |= R_TOKEN_MISMATCH;
          uint64_t k = ((uint64_t)0 << 32) | q;
          if (k < best) best = k;
          if (q < intact) intact = (uint32_t)q;
        }
        if (cl->chain_hash != chain_hash) {
          reasons |= R_TOKEN_MISMATCH;
          if (none_key < best) best = none_key;
        }
        uint32_t na = (uint32_t)cl->footprint.size();
        uint32_t common = n < na ? n : na;
        for (uint32_t j = 0; j < common; ++j) {
          if (fp[j] != cl->footprint[j]) {
            reasons |= R_FOOTPRINT_MISMATCH;
            uint64_t k = ((uint64_t)0 << 32) | j;
            if (k < best) best = k;
            if (j < intact) intact = j;
          }
        }
        if (n != na) {
          reasons |= R_FOOTPRINT_MISMATCH;
          uint64_t k = ((uint64_t)0 << 32) | common;
          if (k < best) best = k;
          if (common < intact) intact = common;
        }
      }
      if (n == 0) {
        reasons |= R_EMPTY;
        if (none_key < best) best = none_key;
      }
      if (n != nt) {
        uint32_t q = (uint32_t)(n < nt ? n : nt);
        reasons |= R_SHAPE_MISMATCH;
        uint64_t k = ((uint64_t)0 << 32) | q;
        if (k < best) best = k;
        if (q < intact) intact = q;
      }
      for (uint32_t j = 0; j < n; ++j) {
        uint32_t b = fp[j];
        if (b >= p->num_blocks) {
          reasons |= R_MISSING_ENTRY;
          uint64_t k = ((uint64_t)0 << 32) | j;
          if (k < best) best = k;
          if (j < intact) intact = j;
        } else if (!cl) {
          /* a claim that was never accepted holds no offload record
           * (NOT_ACCEPTED already says so) */
        } else if (j >= cl->footprint.size() || cl->footprint[j] != b) {
          /* the claim recorded no offload of this block at this position */
          reasons |= R_NO_OFFLOAD_RECORD;
          uint64_t k = ((uint64_t)0 << 32) | j;
          if (k < best) best = k;
          if (j < intact) intact = j;
        } else {
          /* the claim's own record: a failure reported after its offload,
           * or restored bytes whose digest differs from its own */
          bool lf = p->fail_gen[b] > cl->generation;
          bool mm = p->d_res[b] != cl->digest[j];
          if ((lf || mm) && j < intact) intact = j;
          if (j >= pred) {
            /* beyond the predicate: the claimed prefix is intact */
            if (lf || mm) reasons |= R_BEYOND_PREDICATE;
            continue;
          }
          if (lf) reasons |= R_LOAD_FAILED;
          if (mm) reasons |= R_DIGEST_MISMATCH;
          if (lf || mm) {
            uint64_t k = ((uint64_t)1 << 32) | j;
            if (k < best) best = k;
          }
        }
      }
    }

    orc_outcome o;
    std::memset(&o, 0, sizeof(o));
    o.claim_id = ids[c];
    o.num_blocks = n;
    o.reasons = reasons;
    o.intact_blocks = intact;
    o.chain_hash = chain_hash;
    if (best == ~0ull) {
      o.code = OUT_MATERIALIZED;
      o.first_failing_block = kNone;
      o.phys_block = kNone;
    } else {
      uint32_t cls = (uint32_t)(best >> 32);
      uint32_t j = (uint32_t)(best & 0xFFFFFFFFu);
      o.code = cls == 0 ? OUT_UNKNOWN : OUT_RESTORE_FAILED_FAIL_CLOSED;
      o.first_failing_block = j;
      o.phys_block = j < n ? fp[j] : kNone;
      if (cls == 1) {
        o.expected_digest = cl->digest[j];
        o.observed_digest = p->d_res[fp[j]];
      }
      if (j != kNone && j < nt) o.chain_hash_at_fail = h[j];
    }
    out[c] = o;

    if (o.code == OUT_MATERIALIZED) {
      append_event(p, o.claim_id, EV_RESTORED, kNone, kNone, o.chain_hash);
    } else if (o.code == OUT_RESTORE_FAILED_FAIL_CLOSED) {
      append_event(p, o.claim_id, EV_RESTORATION_FAILED, o.first_failing_block, o.phys_block,
                   o.observed_digest);
      append_event(p, o.claim_id, EV_ACTIVE_REQUEST_REFUSED, o.first_failing_block,
                   o.phys_block, o.claim_id);
    } else {
      append_event(p, o.claim_id, EV_OUTCOME_UNKNOWN, o.first_failing_block, o.phys_block,
                   o.reasons);
    }
  }
  return ORC_OK;
}

uint64_t orc_num_events(void* handle) { return static_cast<Pool*>(handle)->log.size(); }

void orc_events(void* handle, orc_event* out) {
  Pool* p = static_cast<Pool*>(handle);
  for (size_t i = 0; i < p->log.size(); ++i) out[i] = p->log[i];
}

/* Drop the events read so far (sequence numbers keep counting). */
void orc_events_clear(void* handle) { static_cast<Pool*>(handle)->log.clear(); }

/* Per-block state: the latest offload digest, the last restored digest,
 * whether some claim recorded the block, and whether a load failure of it
 * has ever been reported. */
void orc_block_state(void* handle, uint64_t* d_off, uint64_t* d_res, uint8_t* valid_off,
                     uint8_t* load_failed) {
  Pool* p = static_cast<Pool*>(handle);
  for (uint32_t b = 0; b < p->num_blocks; ++b) {
    if (d_off) d_off[b] = p->d_off[b];
    if (d_res) d_res[b] = p->d_res[b];
    if (valid_off) valid_off[b] = p->valid_off[b];
    if (load_failed) load_failed[b] = p->fail_gen[b] != 0;
  }
}

/* Lookup (the reuse lookup of section 7, E1, which reports how many of a
 * request's tokens hit offloaded claim footprints).  For each request row,
 * in order: the chain h_0 .. h_{nt-1} of its tokens; hit = the number of
 * leading token blocks whose identity is registered, unambiguous and still
 * held by its block (a block registered since under another identity no
 * longer holds this prefix: the identity is stale and does not hit).  The
 * lookup stops at the first block that is not; if that block's identity is
 * registered but ambiguous (duplicate ownership), the result is UNKNOWN
 * rather than a shorter hit, as is a malformed row (reserved id, or token
 * offsets that run backwards or past the array).  Otherwise HIT when every
 * token block hit (and there is at least one), MISS when none did, PARTIAL
 * in between.  hit_tokens = min(hit * bs, tokens); chain_hash_at_hit =
 * h_{hit-1} (S when hit = 0); last_block = the block registered for
 * h_{hit-1} (NONE when hit = 0).  Block rows are not read.  The registry
 * and event log are not changed. */
int orc_lookup(void* handle, uint32_t num_requests, uint64_t num_tokens, const uint64_t* ids,
               const uint64_t* tok_off, const uint32_t* tokens, orc_lookup_result* out) {
  Pool* p = static_cast<Pool*>(handle);
  for (uint32_t c = 0; c < num_requests; ++c) {
    orc_lookup_result r;
    std::memset(&r, 0, sizeof(r));
    r.request_id = ids[c];
    r.last_block = kNone;
    r.chain_hash_at_hit = p->seed;
    bool bad = ids[c] == kReservedId || tok_off[c] > tok_off[c + 1] ||
               tok_off[c + 1] > num_tokens;
    if (bad) {
      r.status = LK_UNKNOWN;
      out[c] = r;
      continue;
    }
    uint64_t ntok = tok_off[c + 1] - tok_off[c];
    std::vector<uint64_t> h;
    chain(tokens + tok_off[c], ntok, p->block_size, p->seed, &h);
    uint64_t hit = 0;
    bool ambiguous = false;
    while (hit < h.size()) {
      auto it = p->identities.find(h[hit]);
      if (it == p->identities.end()) break;
      if (it->second.ambiguous) {
        ambiguous = true;
        break;
      }
      if (p->holder[it->second.block] != h[hit]) break; /* stale */
      ++hit;
    }
    r.hit_blocks = (uint32_t)hit;
    r.hit_tokens = hit * p->block_size < ntok ? hit * p->block_size : ntok;
    if (hit > 0) {
      r.chain_hash_at_hit = h[hit - 1];
      r.last_block = p->identities[h[hit - 1]].block;
    }
    if (ambiguous)
      r.status = LK_UNKNOWN;
    else if (hit == h.size() && hit > 0)
      r.status = LK_HIT;
    else if (hit == 0)
      r.status = LK_MISS;
    else
      r.status = LK_PARTIAL;
    out[c] = r;
  }
  return ORC_OK;
}

/* Registered identities, and how many of them are ambiguous. */
void orc_identity_stats(void* handle, uint64_t* entries, uint64_t* ambiguous) {
  Pool* p = static_cast<Pool*>(handle);
  uint64_t a = 0;
  for (const auto& kv : p->identities) a += kv.second.ambiguous ? 1 : 0;
  *entries = p->identities.size();
  *ambiguous = a;
}

/* Predicate coverage (leading positions) recorded for a claim at
 * acceptance, or 0xFFFFFFFF if the id is not registered. */
uint32_t orc_claim_predicate(void* handle, uint64_t id) {
  Pool* p = static_cast<Pool*>(handle);
  auto it = p->registry.find(id);
  return it == p->registry.end() ? kNone : it->second.pred_blocks;
}

/* Registry state of one claim id: returns the state bits, or 0 if the id is
 * not registered. */
uint32_t orc_claim_state(void* handle, uint64_t id) {
  Pool* p = static_cast<Pool*>(handle);
  auto it = p->registry.find(id);
  return it == p->registry.end() ? 0 : it->second.state;
}

}  // extern "C"
