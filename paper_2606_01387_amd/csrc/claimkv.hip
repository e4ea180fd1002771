// claimkv.hip -- claim-scoped KV materialization checking for MI355X (gfx950).
//
// HIP kernels and the host side of the C ABI declared in include/claimkv.h.
// The header states what each call computes and which passage of the paper
// ("Fail-Closed Lowering of Resident KV Claims onto LLM Serving Runtimes")
// it follows; this file is the implementation.
//
// Design (one GPU, one stream per pool, all work integer, no MFMA: nothing
// on this path is a dense contraction):
//
//  * Block digest (the HBM-bound stage).  The pool is plane-major
//    [plane][block][chunk].  D(b) = sum_i w_i k_i is linear in the words, so
//    it splits into partial sums over pieces of the canonical block: a piece
//    is one 64-lane x LPW 8-byte-word segment of a plane's chunk (LPW up to
//    24 for whole chunks, 12 KiB; 32 for ragged ones), and since k_i depends
//    only on the word's canonical position, a wave pinned to one piece keeps
//    that piece's keys in VGPRs and streams the same piece of many blocks,
//    with all LPW loads in flight before any use.  The 4 waves of a workgroup take 4 consecutive pieces
//    of the same blocks and park their per-block sums in an LDS ring, which
//    the workgroup adds and writes as one contiguous run of partials; the
//    grid is exactly one resident round, and on larger pools it reads the
//    piece groups in phases (two from 14 GiB, a few piece groups at a time
//    past 32 GiB).  Each 64-bit word costs one
//    32x32->64 multiply-add for lo(w) lo(k) and two 32-bit multiply-adds for
//    the cross terms (only their low 32 bits reach the result mod 2^64).  A
//    small kernel adds each block's partials.  No atomics: results are
//    bitwise deterministic.
//  * Unique blocks.  Blocks referenced by a batch are marked, then compacted
//    in ascending order, so each physical block is read once however many
//    claims alias it.
//  * Claims.  A group of W lanes (W = 2..64, from the batch's mean claim
//    length) owns one claim: lanes take block positions j = j0 + lane.  A
//    window first issues every load that depends only on j (block id, the
//    claim's accepted block, identity and offload digest, the block's
//    tokens), then the block's 16-byte record (restored digest, generation
//    of its latest reported load failure), which stays in flight while the
//    identity step runs; the checks (footprint, identity, missing entry,
//    the claim's own record: a failure reported after its offload or a
//    restored digest different from its own, predicate) follow.  The
//    outcome is the minimum of packed keys (class << 32 | position).
//  * Cache identity.  Offload registers (h_j -> block) of offloaded claims
//    in an open-addressing table with order-independent atomics, and each
//    block remembers the identity of its latest registration; a lookup
//    probes a request's identities block by block and stops at one that is
//    absent, ambiguous, or no longer held by its block.
//  * Events.  Per-claim event counts (0..2) are scanned by one workgroup for
//    batches up to 4096 claims, else in three small kernels (tile sums,
//    one-workgroup scan of the tile sums, write), so the log stays in batch
//    order with no spin waits.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>

#include "claimkv.h"

namespace {

// ------------------------------------------------------------------ constants

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kEmptyId = CLAIM_RESERVED_ID;  // registry empty slot
constexpr uint32_t kNone = CLAIM_NONE;
constexpr uint64_t kNoKey = ~0ull;
constexpr uint64_t kClaimLevelKey = (uint64_t)kNone;  // class 0, position NONE
constexpr uint32_t kMaxBlockSize = 1024;
constexpr int kThreads = 256;
constexpr int kTile = 1024;  // claims per event-scan tile

constexpr uint32_t kStAccepted = 1, kStOffloaded = 2, kStRestoreRequired = 4;

enum MarkMode : int { kMarkAny = 0, kMarkOffloaded = 1, kMarkStaged = 2 };

// --------------------------------------------------------------- hash helpers

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t splitmix_step(uint64_t x) { return mix64(x + kGamma); }

__device__ __forceinline__ uint64_t stream_output(uint64_t s, uint64_t i) {
  return mix64(s + (i + 1) * kGamma);
}

// Slot hash of the claim registry (a data-structure detail, unrelated to the
// digest): the 64-bit finaliser of MurmurHash3.
__device__ __forceinline__ uint64_t slot_of_id(uint64_t id, uint64_t mask) {
  id ^= id >> 33;
  id *= 0xFF51AFD7ED558CCDull;
  id ^= id >> 33;
  id *= 0xC4CEB9FE1A85EC53ull;
  id ^= id >> 33;
  return id & mask;
}

// ----------------------------------------------------------- lane exchange

__device__ __forceinline__ uint32_t lane_read(uint32_t v, uint32_t src_lane) {
  return (uint32_t)__builtin_amdgcn_ds_bpermute((int)(src_lane << 2), (int)v);
}

// Wave-uniform read of lane `lane` (an SGPR index): the result lives in
// SGPRs, so a chain of such values runs on the scalar ALU.
__device__ __forceinline__ uint64_t uniform_read64(uint64_t v, uint32_t lane) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// The claim a group serves.  With one claim per wave (W = 64) the index is
// made provably wave-uniform, so its row is read with scalar loads and its
// chain runs on the scalar ALU.
template <int W>
__device__ __forceinline__ uint64_t group_claim() {
  const uint64_t c = ((uint64_t)blockIdx.x * kThreads + threadIdx.x) / W;
  if constexpr (W == 64) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)c);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(c >> 32));
    return ((uint64_t)hi << 32) | lo;
  }
  return c;
}

__device__ __forceinline__ uint64_t lane_read64(uint64_t v, uint32_t src_lane) {
  const uint32_t lo = lane_read((uint32_t)v, src_lane);
  const uint32_t hi = lane_read((uint32_t)(v >> 32), src_lane);
  return ((uint64_t)hi << 32) | lo;
}


template <int W>
__device__ __forceinline__ uint64_t group_min64(uint64_t v) {
  const uint32_t lane = threadIdx.x & 63;
#pragma unroll
  for (int o = W / 2; o >= 1; o >>= 1) {
    const uint64_t w = lane_read64(v, lane ^ o);
    v = w < v ? w : v;
  }
  return v;
}

// Mask of the calling lane's group (W lanes) whose predicate holds: bit i
// is group lane i.  One ballot instead of a shuffle reduction.
template <int W>
__device__ __forceinline__ uint64_t group_ballot(bool pred) {
  const uint64_t m = __ballot(pred);
  if constexpr (W == 64) {
    return m;
  } else {
    const uint32_t gbase = (threadIdx.x & 63) & ~(uint32_t)(W - 1);
    return (m >> gbase) & ((1ull << W) - 1);
  }
}

// First group lane whose predicate holds, W if none.
template <int W>
__device__ __forceinline__ uint32_t group_first(bool pred) {
  const uint64_t m = group_ballot<W>(pred);
  return m ? (uint32_t)__builtin_ctzll(m) : (uint32_t)W;
}

// Value of group lane i.  With one group per wave i is wave-uniform and a
// readlane serves; narrower groups read through the LDS crossbar.
template <int W>
__device__ __forceinline__ uint64_t group_read64(uint64_t v, uint32_t gbase, uint32_t i) {
  if constexpr (W == 64) {
    return uniform_read64(v, i);
  } else {
    return lane_read64(v, gbase + i);
  }
}

// The previous lane's value (lane 0 gets 0): a DPP shift of the whole wave
// by one lane, which callers override at the first lane of each group.
__device__ __forceinline__ uint64_t prev_lane64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)v, 0x138, 0xf, 0xf, false);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(v >> 32), 0x138, 0xf, 0xf, false);
  return ((uint64_t)hi << 32) | lo;
}

template <int W>
__device__ __forceinline__ uint32_t group_or(uint32_t v) {
  const uint32_t lane = threadIdx.x & 63;
#pragma unroll
  for (int o = W / 2; o >= 1; o >>= 1) v |= lane_read(v, lane ^ o);
  return v;
}

// ---------------------------------------------------------- kernel argument

struct BatchDev {
  uint64_t C, N, T;
  const uint64_t* ids;
  const uint32_t* bo;
  const uint32_t* bi;
  const uint64_t* to;
  const uint32_t* tok;
  const uint64_t* pred;  // predicate tokens per claim, or null
};

struct RegEntry {  // one 64-byte line per slot: a probe touches one line
  uint64_t key;     // claim id; kEmptyId marks an empty slot
  uint32_t state;   // kSt* bits
  uint32_t nblk;    // accepted block-table entries
  uint64_t ntok;    // accepted token count
  uint64_t chain;   // accepted chain hash h_{nt-1}
  uint64_t fpoff;   // accepted footprint: fp[fpoff .. fpoff + nblk)
  uint32_t pred;    // leading positions the accepted predicate covers
  uint32_t pad0;
  uint64_t gen;     // generation of the claim's offload
  uint64_t pad1;
};

struct RegDev {
  uint64_t mask;
  RegEntry* e;
  const uint32_t* fp;
  uint64_t* idn;  // accepted identities h_j, at the footprint's offsets
  uint64_t* dig;  // the claim's own offload digest of the block at each position
};

// Per-block record the check reads at every block position (one 16-byte
// load): the block's restored digest as of the last check that digested
// it, and the generation of its latest reported load failure (0: none).
struct BlockRes {
  uint64_t d_res;
  uint64_t fail_gen;
};

// Cache-identity table: open addressing on the identity h_j, linear
// probing, key 0 marks an empty slot (the identity 0 itself lives in the
// extra entry e[mask + 1]).  block is the first block registered for the
// identity; kIdAmbiguous is set once a different block is registered too.
constexpr uint32_t kIdUsed = 1u, kIdAmbiguous = 2u;

struct IdEntry {
  uint64_t key;
  uint32_t block;  // kNone until the first registration
  uint32_t flags;  // kIdUsed | kIdAmbiguous
};

// Where the first claim that registered an identity keeps its accepted
// identities: the identity store index of the identity itself, and one past
// that claim's last accepted identity.  A lookup that reaches the identity
// follows that claim's identities to confirm many positions at once.
struct IdSrc {
  uint64_t at;
  uint64_t end;
};

struct IdDev {
  uint64_t mask;
  IdEntry* e;  // mask + 2 entries
  IdSrc* src;  // mask + 2 entries, parallel to e
};

struct Pend {  // events a claim will append (0..2), written before the scan
  uint64_t aux0, aux1;
  uint32_t kinds;  // kind0 | kind1 << 8
  uint32_t j;
  uint32_t phys;
  uint32_t pad;
};

struct Counters {  // device-resident counters of one pool (72 bytes)
  uint32_t uniq_count;
  uint32_t dup_flag;      // kFlagDupId | kFlagBackwardRow
  uint64_t log_count;     // events held in the log
  uint64_t seq_next;      // next global sequence number
  uint64_t call_pos;      // log position of the current call's first event (kDropped: none)
  uint64_t call_seq;      // its sequence number
  uint64_t reg_count;     // claims registered
  uint64_t id_entries;    // identities registered
  uint64_t id_ambiguous;  // identities registered to two or more blocks
  uint32_t log_dropped;   // a call's events did not fit the log and were dropped
  uint32_t pad;
};

static_assert(sizeof(Counters) == 72, "Counters layout");

// call_pos of a call whose events do not fit the log: they are dropped, all
// of them, and log_dropped is set.  The host bounds every call it queues
// itself; the device bound keeps the log in bounds for work the host cannot
// see (a captured graph replayed).
constexpr uint64_t kDropped = ~0ull;

// dup_flag bits set by k_dupcheck: a claim id occurs twice or is already
// registered (the batch is refused); some block row runs backwards, so the
// rows after it may share block-table entries with earlier rows.
constexpr uint32_t kFlagDupId = 1, kFlagBackwardRow = 2;

// Where claim c's accepted footprint and identities start in the stores:
// at its own block-table offset when the batch's rows are disjoint, else
// at the offset k_footprint_offsets gave it.
__device__ __forceinline__ uint64_t store_at(const uint64_t* fpo, uint64_t fp_base, uint64_t c,
                                             uint32_t bo0) {
  return fpo ? fpo[c] : fp_base + bo0;
}
static_assert(sizeof(IdEntry) == 16, "IdEntry layout");
static_assert(sizeof(claim_lookup_result) == 40, "claim_lookup_result layout");
static_assert(sizeof(claim_outcome) == 64, "claim_outcome layout");
static_assert(sizeof(claim_event) == 40, "claim_event layout");
static_assert(sizeof(Pend) == 32, "Pend layout");
static_assert(sizeof(RegEntry) == 64, "RegEntry layout");
static_assert(sizeof(BlockRes) == 16, "BlockRes layout");

struct Row {
  uint64_t id;
  uint64_t to0, ntok;
  uint32_t bo0, n;
  bool malformed;
};

__device__ __forceinline__ Row read_row(const BatchDev& b, uint64_t c) {
  Row r;
  r.id = b.ids[c];
  const uint32_t bo0 = b.bo[c], bo1 = b.bo[c + 1];
  const uint64_t to0 = b.to[c], to1 = b.to[c + 1];
  r.malformed = r.id == kEmptyId || bo0 > bo1 || (uint64_t)bo1 > b.N || to0 > to1 || to1 > b.T;
  r.bo0 = bo0;
  r.n = r.malformed ? 0 : bo1 - bo0;
  r.to0 = to0;
  r.ntok = r.malformed ? 0 : to1 - to0;
  return r;
}

__device__ __forceinline__ int64_t reg_find(const RegDev& r, uint64_t id) {
  if (id == kEmptyId) return -1;
  uint64_t s = slot_of_id(id, r.mask);
  for (uint64_t probe = 0; probe <= r.mask; ++probe) {
    const uint64_t k = r.e[s].key;
    if (k == id) return (int64_t)s;
    if (k == kEmptyId) return -1;
    s = (s + 1) & r.mask;
  }
  return -1;
}

// Registration of an identity happens in two passes, so that a position
// whose identity is already present costs no atomic and a new identity one.
//
// Pass 1 (id_insert, during acceptance): find the identity's slot, reading
// before writing; only an empty slot is claimed, with one CAS on the key.
// The CAS winner stores the block and where its claim keeps its accepted
// identities (IdSrc) with plain stores.  The identity 0 lives in the extra
// entry e[mask + 1], claimed by setting kIdUsed.
//
// Pass 2 (k_register_owners, after acceptance): every registering position
// compares its block with the stored one; a different block is duplicate
// ownership and marks the identity ambiguous for good.  Among racing first
// registrants the stored block and source depend on the order, but they
// are read only for identities that are not ambiguous, so every output is
// order-independent.
//
// Returns kRegNewEntry if this call inserted the identity.
constexpr uint32_t kRegNewEntry = 1;

__device__ uint32_t id_insert(const IdDev& t, uint64_t key, uint32_t block, uint64_t at,
                              uint64_t end) {
  uint64_t s;
  if (key == 0) {
    s = t.mask + 1;
    if (atomicOr(&t.e[s].flags, kIdUsed) & kIdUsed) return 0;
  } else {
    s = slot_of_id(key, t.mask);
    for (uint64_t probe = 0;; ++probe) {
      if (probe > t.mask) return 0;  // unreachable: the table is at most half full
      // keys only ever go from 0 to their final value, so a non-zero read is
      // final; a stale 0 only costs a CAS that reports the real key
      uint64_t k = t.e[s].key;
      if (k == 0)
        k = atomicCAS((unsigned long long*)&t.e[s].key, 0ull, (unsigned long long)key);
      if (k == 0) break;         // inserted here
      if (k == key) return 0;    // present
      s = (s + 1) & t.mask;      // another identity: keep probing
    }
  }
  t.e[s].block = block;
  t.src[s].at = at;
  t.src[s].end = end;
  return kRegNewEntry;
}

// Adds the active lanes whose predicate holds to *counter with one atomic
// per wave (many lanes adding 1 to one address serialize on it).  Every
// active lane must call it at the same point.
__device__ __forceinline__ void wave_count(uint64_t* counter, bool pred) {
  const uint64_t m = __ballot(pred);
  const uint64_t active = __ballot(true);
  if (m && (threadIdx.x & 63) == (uint32_t)__builtin_ctzll(active))
    atomicAdd((unsigned long long*)counter, (unsigned long long)__builtin_popcountll(m));
}

__device__ __forceinline__ const IdEntry* id_find(const IdDev& t, uint64_t key) {
  if (key == 0) {
    const IdEntry* e = t.e + t.mask + 1;
    return (e->flags & kIdUsed) ? e : nullptr;
  }
  uint64_t s = slot_of_id(key, t.mask);
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    const uint64_t k = t.e[s].key;
    if (k == key) return t.e + s;
    if (k == 0) return nullptr;
    s = (s + 1) & t.mask;
  }
  return nullptr;
}

// Token multilinear of one token block, sum over its tokens of tok * t_m.
// kDepth 2: the loads of a full 16-token chunk are issued together and the
// next chunk is in flight while the current one is summed (wide groups:
// few, long claims, where latency rules).  kDepth 1: 16-token chunks loaded
// together, one after another (16 registers: narrow groups of the check).
// kDepth 0: a plain loop (fewest registers: narrow lookups and
// acceptance, where occupancy rules).  The tail of a partial block goes
// token by token.
template <int kDepth>
__device__ __forceinline__ uint64_t block_multilinear(const uint32_t* __restrict__ tok,
                                                      uint64_t first, uint64_t count,
                                                      const uint64_t* tkey) {
  constexpr int kChunk = 16;
  uint64_t m_sum = 0, m = 0;
  if constexpr (kDepth == 0) {
    for (; m < count; ++m) m_sum += (uint64_t)tok[first + m] * tkey[m];
    return m_sum;
  } else if constexpr (kDepth == 1) {
    for (; m + kChunk <= count; m += kChunk) {
      uint32_t cur[kChunk];
#pragma unroll
      for (int k = 0; k < kChunk; ++k) cur[k] = tok[first + m + k];
#pragma unroll
      for (int k = 0; k < kChunk; ++k) m_sum += (uint64_t)cur[k] * tkey[m + k];
    }
  } else if (count >= kChunk) {
    uint32_t cur[kChunk];
#pragma unroll
    for (int k = 0; k < kChunk; ++k) cur[k] = tok[first + k];
    for (; m + kChunk <= count; m += kChunk) {
      const bool more = m + 2 * kChunk <= count;
      uint32_t nxt[kChunk];
      if (more) {
#pragma unroll
        for (int k = 0; k < kChunk; ++k) nxt[k] = tok[first + m + kChunk + k];
      }
#pragma unroll
      for (int k = 0; k < kChunk; ++k) m_sum += (uint64_t)cur[k] * tkey[m + k];
      if (more) {
#pragma unroll
        for (int k = 0; k < kChunk; ++k) cur[k] = nxt[k];
      }
    }
  }
  for (; m < count; ++m) m_sum += (uint64_t)tok[first + m] * tkey[m];
  return m_sum;
}

// First 16-token chunk of a block, loaded ahead (count < 16: not loaded;
// the block's multilinear then loads its tokens itself).
__device__ __forceinline__ void prefetch_chunk(uint32_t (&ch)[16], const uint32_t* __restrict__ tok,
                                               uint64_t first, uint64_t count) {
  if (count >= 16) {
#pragma unroll
    for (int k = 0; k < 16; ++k) ch[k] = tok[first + k];
  }
}

// Token multilinear of a block whose first 16-token chunk, if it has one,
// was loaded ahead into ch; the rest of a longer block is summed with
// block_multilinear<kTail>.
template <int kTail>
__device__ __forceinline__ uint64_t multilinear_prefetched(const uint32_t (&ch)[16],
                                                          const uint32_t* __restrict__ tok,
                                                          uint64_t first, uint64_t count,
                                                          const uint64_t* tkey) {
  if (count < 16) return block_multilinear<0>(tok, first, count, tkey);
  uint64_t m_sum = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) m_sum += (uint64_t)ch[k] * tkey[k];
  if (count > 16) m_sum += block_multilinear<kTail>(tok, first + 16, count - 16, tkey + 16);
  return m_sum;
}

// Put the wave-uniform value `val` into lane `lane` of `old` (v_writelane;
// the lane select goes through M0, written by a scalar move, so the
// instruction reads one scalar register besides it).
__device__ __forceinline__ uint32_t write_lane(uint32_t old, uint32_t val, uint32_t lane) {
  asm("v_writelane_b32 %0, %1, m0" : "+v"(old) : "s"(val), "{m0}"(lane));
  return old;
}

// Chain steps t < steps of one window: h advances through the group's
// multilinears, and lane t of the group keeps h_{j0 + t}.
template <int W>
__device__ __forceinline__ uint64_t chain_window(uint64_t& h, uint64_t m_sum, uint32_t gl,
                                                 uint32_t gbase, uint64_t steps) {
  if constexpr (W == 64) {  // one claim per wave: the chain runs on the scalar ALU
    // h is the same in every lane; say so, so that it lives in SGPRs
    // (the builtin returns int: widen through uint32_t, never by sign extension)
    const uint32_t h_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)h);
    const uint32_t h_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(h >> 32));
    h = ((uint64_t)h_hi << 32) | h_lo;
    uint32_t lo = 0, hi = 0;
    for (uint32_t t = 0; t < steps; ++t) {
      h = splitmix_step(h ^ uniform_read64(m_sum, t));
      lo = write_lane(lo, (uint32_t)h, t);
      hi = write_lane(hi, (uint32_t)(h >> 32), t);
    }
    return ((uint64_t)hi << 32) | lo;
  } else {
    uint64_t my_h = 0;
    for (uint32_t t = 0; t < steps; ++t) {
      h = splitmix_step(h ^ lane_read64(m_sum, gbase + t));
      if (gl == t) my_h = h;
    }
    return my_h;
  }
}

__device__ __forceinline__ void load_token_keys(uint64_t* tkey, uint32_t bs, uint64_t seed) {
  for (uint32_t m = threadIdx.x; m < bs; m += blockDim.x) tkey[m] = stream_output(~seed, m) | 1ull;
  __syncthreads();
}

// ------------------------------------------------------------ small kernels

template <typename T>
__global__ void __launch_bounds__(kThreads) k_fill(T* p, uint64_t n, T v) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

__global__ void __launch_bounds__(kThreads) k_fill_strided(uint64_t* p, uint64_t n,
                                                           uint32_t stride_words, uint64_t v) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i * stride_words] = v;
}

// Mark the in-range blocks referenced by well-formed claims (filtered by
// mode).  A group of W lanes walks one claim's row.
template <int W>
__global__ void __launch_bounds__(kThreads) k_mark(BatchDev b, uint32_t nb, int mode,
                                                   const uint8_t* __restrict__ valid_off,
                                                   const uint32_t* __restrict__ slot_of,
                                                   uint8_t* __restrict__ mark) {
  const uint64_t c = group_claim<W>();
  if (c >= b.C) return;
  const uint32_t gl = threadIdx.x & (W - 1);
  const Row r = read_row(b, c);
  for (uint32_t j = gl; j < r.n; j += W) {
    const uint32_t blk = b.bi[(uint64_t)r.bo0 + j];
    if (blk >= nb) continue;
    if (mode == kMarkOffloaded && !valid_off[blk]) continue;
    if (mode == kMarkStaged && slot_of[blk] == kNone) continue;
    // most blocks are referenced many times: read before writing, so that
    // the stores (all of the same value) stay about one per block
    if (!mark[blk]) mark[blk] = 1;
  }
}

// Exclusive scan over a 1024-thread workgroup; returns the prefix and
// writes the total to *total.
__device__ uint32_t block_exclusive_scan_1024(uint32_t v, uint32_t* total, uint32_t* lds16) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t up = lane_read(incl, lane >= (uint32_t)o ? lane - o : lane);
    if (lane >= (uint32_t)o) incl += up;
  }
  if (lane == 63) lds16[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < 16; ++w) {
      const uint32_t t = lds16[w];
      lds16[w] = run;
      run += t;
    }
    lds16[16] = run;
  }
  __syncthreads();
  const uint32_t out = lds16[wave] + incl - v;
  *total = lds16[16];
  __syncthreads();
  return out;
}

// Ordered compaction of the marks into the unique-block list (ascending
// block id).  One workgroup of 1024 threads, 8 marks per thread per step
// read as one 8-byte word (the mark array is padded to a multiple of 16
// bytes with zeros); a step's indices are gathered in LDS and written out
// with coalesced stores; clears the marks it reads.
__global__ void __launch_bounds__(1024) k_compact(uint8_t* __restrict__ mark, uint32_t nb,
                                                  uint32_t* __restrict__ uniq,
                                                  Counters* __restrict__ ctr) {
  constexpr uint32_t kPer = 8;
  __shared__ uint32_t lds[17];
  __shared__ uint32_t out[1024 * kPer];
  uint32_t base = 0;
  const uint64_t padded = ((uint64_t)nb + 15) / 16 * 16;
  for (uint64_t t0 = 0; t0 < padded; t0 += 1024ull * kPer) {
    const uint64_t first = t0 + (uint64_t)threadIdx.x * kPer;
    uint32_t bits = 0;
    if (first < padded) {
      const uint2 m = *(const uint2*)(mark + first);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (((k < 4 ? m.x : m.y) >> (8 * (k % 4))) & 0xFFu) bits |= 1u << k;
    }
    uint32_t total;
    uint32_t pos = block_exclusive_scan_1024(__builtin_popcount(bits), &total, lds);
    if (bits) {
      for (uint32_t k = 0; k < kPer; ++k)
        if (bits & (1u << k)) out[pos++] = (uint32_t)(first + k);
      *(uint2*)(mark + first) = make_uint2(0u, 0u);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < total; i += 1024) uniq[base + i] = out[i];
    base += total;
    __syncthreads();
  }
  if (threadIdx.x == 0) ctr->uniq_count = base;
}

// ----------------------------------------------------------- digest kernel

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Partial digests of the unique blocks.
//
// A piece is one 64-lane x LPW-word segment of a plane's chunk (piece index
// ps = plane * segs + segment).  Workgroup (piece group pg, group g) runs 4
// waves on the 4 consecutive pieces 4pg .. 4pg+3 of the same blocks
// u = g, g + groups, g + 2 groups, ...  Only pga piece groups are read at a
// time (pga divides the piece-group count): workgroup blockIdx takes piece
// groups pgl, pgl + pga, pgl + 2 pga, ... in turn (pgl = blockIdx % pga,
// g = blockIdx / pga), each one a phase over its blocks, so every workgroup
// runs the same number of phases.  Lane l, slot k of a wave covers the
// 64-bit word q = s*64*LPW + 64k + l of the plane's chunk, canonical word
// i = p*CW + q, whose key it keeps in VGPRs.  Each load instruction moves
// 512 contiguous bytes (8 per lane); 8-byte loads measured about 2 % faster
// than 16-byte loads at the same bytes in flight per wave.
// Each wave's per-block sum goes to an LDS ring; when the ring is full (or
// the blocks run out) the workgroup adds its 4 rings and writes one
// contiguous run of per-(piece group, block) partials,
//   partial[(pg * groups + g) * NW + n],  NW = ceil(U / groups),
// so the streaming reads are not interleaved with scattered small writes.
// (Giving the 4 waves the same piece of 4 adjacent blocks instead, which
// reads whole runs of adjacent chunks when a chunk is one piece, measured
// about 1 % slower on 16 KiB chunks.)
// Optionally copies the words to staging ([slot][plane][chunk], slot =
// unique index).
constexpr int kRing = 256;

__device__ __forceinline__ uint64_t dpp_wave_sum64(uint64_t v) {
  // Out-of-row sources read 0 (old = 0): after row shifts by 1, 2, 4 and 8
  // lane 15 of every row holds its row's total, and the two row broadcasts
  // fold the rows into lane 63.
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#define DPP_STEP(ctrl, row_mask)                                                       \
  {                                                                                    \
    const uint32_t l2 = __builtin_amdgcn_update_dpp(0u, lo, ctrl, row_mask, 0xf, false); \
    const uint32_t h2 = __builtin_amdgcn_update_dpp(0u, hi, ctrl, row_mask, 0xf, false); \
    const uint64_t t = (((uint64_t)hi << 32) | lo) + (((uint64_t)h2 << 32) | l2);       \
    lo = (uint32_t)t;                                                                  \
    hi = (uint32_t)(t >> 32);                                                          \
  }
  DPP_STEP(0x111, 0xf)  // row_shr:1
  DPP_STEP(0x112, 0xf)  // row_shr:2
  DPP_STEP(0x114, 0xf)  // row_shr:4
  DPP_STEP(0x118, 0xf)  // row_shr:8
  DPP_STEP(0x142, 0xa)  // row_bcast:15 into rows 1 and 3
  DPP_STEP(0x143, 0xc)  // row_bcast:31 into rows 2 and 3
#undef DPP_STEP
  const uint32_t l = __builtin_amdgcn_readlane(lo, 63), h = __builtin_amdgcn_readlane(hi, 63);
  return ((uint64_t)h << 32) | l;
}

// RAGGED: the chunk's last segment is partly past its end (masked slots).
// STAGE: also copy the words to staging (offload with staging).
// Position of a pool word in its block's full canonical bytes: the index of
// its key.  A pool that holds every head has word q of plane p's chunk at
// p * chunk_words + q.  A head shard (tensor parallel by KV head) holds heads
// [first, first + heads) of blocks with `total` heads: its chunk is rows
// r = t * heads + h ([token][head]) of row_words words, and row r sits at
// row t * total + first + h of the full chunk.  So a shard's digest is the
// full digest's sum over the shard's words, and shards add up to it.
struct KeyMap {
  uint32_t chunk_words;  // this pool's chunk
  uint32_t row_words;    // one head's words of one token (shards only)
  uint32_t heads, total, first;
  __device__ __forceinline__ uint64_t at(uint32_t p, uint32_t q) const {
    if (heads == total) return (uint64_t)p * chunk_words + q;
    const uint32_t r = q / row_words, w = q - r * row_words;
    const uint32_t t = r / heads, h = r - t * heads;
    const uint64_t full_chunk = (uint64_t)(chunk_words / heads) * total;
    return (uint64_t)p * full_chunk + ((uint64_t)t * total + first + h) * row_words + w;
  }
};

template <int LPW, bool RAGGED, bool STAGE>
__global__ void __launch_bounds__(kThreads) k_digest(const u32x2* __restrict__ pool, uint32_t nb,
                                                     uint32_t chunk_words, uint32_t planes,
                                                     uint32_t segs, uint32_t pga, uint32_t groups,
                                                     const uint32_t* __restrict__ uniq,
                                                     const Counters* __restrict__ ctr,
                                                     uint64_t seed, KeyMap km,
                                                     uint64_t* __restrict__ partial,
                                                     u32x2* __restrict__ staging) {
  __shared__ uint64_t ring[kThreads / 64][kRing];
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t ps_total = planes * segs;
  const uint32_t pgs = (ps_total + 3) / 4;
  const uint32_t g = blockIdx.x / pga;
  if (g >= groups) return;
  const uint32_t U = ctr->uniq_count;
  const uint32_t NW = (U + groups - 1) / groups;
  for (uint32_t pg = blockIdx.x % pga; pg < pgs; pg += pga) {  // one phase per piece group
    const uint32_t ps = pg * 4 + w;
    const bool active = ps < ps_total;  // wave-uniform: the last piece group may be short
    const uint32_t p = active ? ps / segs : 0, s = active ? ps % segs : 0;
    const uint32_t q0 = s * 64u * LPW + lane;  // this lane's word in slot 0

    uint32_t klo[LPW], khi[LPW];
#pragma unroll
    for (int k = 0; k < LPW; ++k) {
      const uint32_t q = q0 + 64u * k;
      const uint64_t key = stream_output(seed, km.at(p, q)) | 1ull;
      const bool ok = !RAGGED || q < chunk_words;
      klo[k] = ok ? (uint32_t)key : 0u;  // a masked slot contributes 0
      khi[k] = ok ? (uint32_t)(key >> 32) : 0u;
    }

    const u32x2* plane = pool + (uint64_t)p * nb * chunk_words;
    uint32_t n = 0;
    for (uint32_t u = g; u < U; u += groups, ++n) {
      uint64_t sum = 0;
      if (active) {
        const u32x2* chunk = plane + (uint64_t)uniq[u] * chunk_words;
        const u32x2* lanep = chunk + q0;  // slot k at lanep + 64k: immediate offsets
        u32x2 x[LPW];
#pragma unroll
        for (int k = 0; k < LPW; ++k) {
          // a masked slot reads the chunk's first word (its key is 0): no
          // address outside the chunk is ever formed
          if (!RAGGED || q0 + 64u * k < chunk_words)
            x[k] = __builtin_nontemporal_load(lanep + 64 * k);
          else
            x[k] = __builtin_nontemporal_load(chunk);
        }
        __builtin_amdgcn_sched_barrier(0);  // every load in flight before any use
        uint64_t acc = 0;
        uint32_t cross = 0;
#pragma unroll
        for (int k = 0; k < LPW; ++k) {
          // word = (x.y:x.x); only the low 32 bits of the cross terms reach
          // the product mod 2^64
          acc += (uint64_t)x[k].x * klo[k];
          cross += x[k].x * khi[k] + x[k].y * klo[k];
        }
        sum = dpp_wave_sum64(acc + ((uint64_t)cross << 32));
        if constexpr (STAGE) {
          u32x2* dst = staging + ((uint64_t)u * planes + p) * chunk_words + q0;
#pragma unroll
          for (int k = 0; k < LPW; ++k)
            if (!RAGGED || q0 + 64u * k < chunk_words) dst[64 * k] = x[k];
        }
      }
      const uint32_t slot = n % kRing;
      if (lane == 0) ring[w][slot] = sum;
      if (slot == kRing - 1 || u + groups >= U) {  // the same for all 4 waves
        __syncthreads();
        const uint32_t n0 = n - slot;
        for (uint32_t i = threadIdx.x; i <= slot; i += kThreads)
          partial[((uint64_t)pg * groups + g) * NW + n0 + i] =
              ring[0][i] + ring[1][i] + ring[2][i] + ring[3][i];
        __syncthreads();
      }
    }
  }
}

// Add each unique block's piece-group partials.
//   mode 0 (offload): d_off (the latest offload's digest), valid_off = 1
//                     (some claim records the block), slot_of: the
//                     block's staging slot slot0 + u when staged, else none
//                     (an unstaged offload drops the block's staged copy)
//   mode 1 (check):   the restored digest in the block's record; every
//                     block whose record a check's claims compare is one
//                     of its unique blocks, so the claim stage reads only
//                     digests written here
__global__ void __launch_bounds__(kThreads) k_finalize(const uint32_t* __restrict__ uniq,
                                                       const Counters* __restrict__ ctr,
                                                       const uint64_t* __restrict__ partial,
                                                       uint32_t pgs, uint32_t groups, int mode,
                                                       int staged, uint32_t slot0,
                                                       uint64_t* __restrict__ d_off,
                                                       uint8_t* __restrict__ valid_off,
                                                       uint32_t* __restrict__ slot_of,
                                                       BlockRes* __restrict__ bres) {
  // One lane per unique block.  Unique index u = n * groups + g was digested
  // by the workgroups of group g, which wrote its partials at
  // partial[(pg * groups + g) * NW + n]; slot t = g * NW + n puts
  // consecutive n of one group in consecutive lanes, so each piece group's
  // partials are read as one contiguous run per wave.
  const uint32_t U = ctr->uniq_count;
  const uint32_t NW = (U + groups - 1) / groups;
  const uint64_t slots = (uint64_t)groups * NW;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads;
  for (uint64_t t = (uint64_t)blockIdx.x * kThreads + threadIdx.x; t < slots; t += stride) {
    const uint32_t g = (uint32_t)(t / NW), n = (uint32_t)(t % NW);
    const uint32_t u = n * groups + g;
    if (u >= U) continue;
    // partials in batches of 32 loads issued together
    const uint64_t* src = partial + (uint64_t)g * NW + n;
    const uint64_t pstride = (uint64_t)groups * NW;
    uint64_t sum = 0;
    for (uint32_t pg0 = 0; pg0 < pgs; pg0 += 32) {
      uint64_t v[32];
#pragma unroll
      for (uint32_t k = 0; k < 32; ++k) v[k] = pg0 + k < pgs ? src[(uint64_t)(pg0 + k) * pstride] : 0ull;
#pragma unroll
      for (uint32_t k = 0; k < 32; ++k) sum += v[k];
    }
    const uint32_t b = uniq[u];
    if (mode == 0) {
      d_off[b] = sum;
      valid_off[b] = 1;
      slot_of[b] = staged ? slot0 + u : kNone;
    } else {
      bres[b].d_res = sum;
    }
  }
}

// ----------------------------------------------------------------- offload

// Duplicate ownership: a non-reserved id occurring twice in the batch or
// already registered sets kFlagDupId; a block row that runs backwards sets
// kFlagBackwardRow.  table is a cleared scratch hash set.
__global__ void __launch_bounds__(kThreads) k_dupcheck(BatchDev b, RegDev reg,
                                                       unsigned long long* table, uint64_t tmask,
                                                       Counters* ctr) {
  const uint64_t c = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
  if (c >= b.C) return;
  if (b.bo[c + 1] < b.bo[c]) atomicOr(&ctr->dup_flag, kFlagBackwardRow);
  const uint64_t id = b.ids[c];
  if (id == kEmptyId) return;
  if (reg_find(reg, id) >= 0) {
    atomicOr(&ctr->dup_flag, kFlagDupId);
    return;
  }
  uint64_t s = slot_of_id(id, tmask);
  for (uint64_t probe = 0; probe <= tmask; ++probe) {
    const unsigned long long old = atomicCAS(table + s, (unsigned long long)kEmptyId,
                                             (unsigned long long)id);
    if (old == kEmptyId) return;
    if (old == id) {
      atomicOr(&ctr->dup_flag, kFlagDupId);
      return;
    }
    s = (s + 1) & tmask;
  }
}

// Store offsets for a batch whose block rows may share entries (some row
// runs backwards): each well-formed claim gets a run of its own in the
// footprint and identity stores, at fp_base plus the exclusive prefix sum of
// the row lengths in claim order (a malformed row takes none); fpo[C] is the
// total.  One workgroup; only such batches pay for it.
__global__ void __launch_bounds__(1024) k_footprint_offsets(BatchDev b, uint64_t fp_base,
                                                            uint64_t* __restrict__ fpo) {
  __shared__ uint64_t s_sum[1024];
  const uint32_t t = threadIdx.x;
  const uint64_t per = (b.C + 1023) / 1024;
  const uint64_t c0 = (uint64_t)t * per < b.C ? (uint64_t)t * per : b.C;
  const uint64_t c1 = c0 + per < b.C ? c0 + per : b.C;
  uint64_t mine = 0;
  for (uint64_t c = c0; c < c1; ++c) mine += read_row(b, c).n;
  s_sum[t] = mine;
  __syncthreads();
  for (uint32_t d = 1; d < 1024; d <<= 1) {  // inclusive scan of the 1024 sums
    const uint64_t v = t >= d ? s_sum[t - d] : 0;
    __syncthreads();
    s_sum[t] += v;
    __syncthreads();
  }
  uint64_t at = fp_base + s_sum[t] - mine;
  for (uint64_t c = c0; c < c1; ++c) {
    fpo[c] = at;
    at += read_row(b, c).n;
  }
  if (t == 1023) fpo[b.C] = s_sum[1023];
}

// Acceptance: chain hash of the claim's tokens, presence of its footprint
// (stored as the accepted footprint, with the claim's own offload digest of
// each in-range block: the offload digest ran before acceptance), its
// accepted identities and their registration, and the record of its
// ACCEPTED (+ OFFLOADED) events.
template <int W>
__global__ void __launch_bounds__(kThreads) k_accept(BatchDev b, RegDev reg, IdDev ids,
                                                     uint32_t nb, uint32_t bs, uint64_t seed,
                                                     uint64_t fp_base,
                                                     const uint64_t* __restrict__ fpo,
                                                     const uint64_t* __restrict__ d_off,
                                                     uint32_t* __restrict__ fp_out,
                                                     Counters* __restrict__ ctr,
                                                     uint32_t* __restrict__ cnt,
                                                     Pend* __restrict__ pend, uint64_t c_lo,
                                                     uint64_t c_hi) {
  __shared__ uint64_t tkey[kMaxBlockSize];
  load_token_keys(tkey, bs, seed);
  const uint64_t c = c_lo + group_claim<W>();  // claims [c_lo, c_hi) of the batch
  if (c >= c_hi) return;
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t gl = lane & (W - 1), gbase = lane & ~(uint32_t)(W - 1);
  const Row r = read_row(b, c);
  const uint64_t nt = (r.ntok + bs - 1) / bs;

  const uint64_t at0 = r.malformed ? 0 : store_at(fpo, fp_base, c, r.bo0);
  // presence first: only an offloaded claim registers its identities
  uint32_t missing = 0;
  for (uint64_t j = gl; j < r.n; j += W) {
    const uint32_t blk = b.bi[(uint64_t)r.bo0 + j];
    fp_out[at0 + j] = blk;  // the accepted footprint
    reg.dig[at0 + j] = blk < nb ? d_off[blk] : 0ull;  // and the claim's own offload record
    if (blk >= nb) missing = 1;
  }
  missing = group_or<W>(missing);
  const bool offloaded = !r.malformed && r.n > 0 && !missing && (uint64_t)r.n == nt;
  const uint64_t npos = (uint64_t)r.n < nt ? (uint64_t)r.n : nt;  // positions with block and tokens

  uint64_t h = seed;
  for (uint64_t j0 = 0; j0 < nt; j0 += W) {
    const uint64_t j = j0 + gl;
    uint64_t m_sum = 0;
    if (j < nt) {
      const uint64_t first = j * bs;
      const uint64_t count = r.ntok - first < bs ? r.ntok - first : bs;
      m_sum = block_multilinear<(W >= 16 ? 2 : 0)>(b.tok, r.to0 + first, count, tkey);
    }
    const uint64_t steps = nt - j0 < (uint64_t)W ? nt - j0 : (uint64_t)W;
    const uint64_t my_h = chain_window<W>(h, m_sum, gl, gbase, steps);
    uint32_t res = 0;
    if (j < npos) {
      reg.idn[at0 + j] = my_h;
      if (offloaded) res = id_insert(ids, my_h, b.bi[(uint64_t)r.bo0 + j], at0 + j, at0 + npos);
    }
    wave_count(&ctr->id_entries, res & kRegNewEntry);
  }
  if (gl != 0) return;
  if (r.malformed) {
    cnt[c] = 0;
    return;
  }
  // the claim is registered by k_register_claims, one lane per claim, from
  // this record (its chain hash and whether it was offloaded)
  Pend pe;
  pe.aux0 = h;
  pe.aux1 = r.n;
  pe.kinds = CLAIM_EV_ACCEPTED | (offloaded ? (CLAIM_EV_OFFLOADED << 8) : 0u);
  pe.j = kNone;
  pe.phys = kNone;
  pe.pad = 0;
  pend[c] = pe;
  cnt[c] = offloaded ? 2 : 1;
}

// Registration of the batch's claims in the registry, one lane per claim,
// after acceptance: a read of each probed slot first, then one CAS on the
// key of an empty one (the batch's ids are distinct and none is registered,
// which the duplicate check established, so a lost CAS only means another
// claim took the slot).  Kept out of the claim-group kernel so that each
// wave waits on its atomics once, for 64 claims.
__global__ void __launch_bounds__(kThreads) k_register_claims(BatchDev b, RegDev reg, uint32_t bs,
                                                              uint64_t fp_base, uint64_t gen,
                                                              const uint64_t* __restrict__ fpo,
                                                              const Pend* __restrict__ pend,
                                                              Counters* __restrict__ ctr) {
  const uint64_t c = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
  bool inserted = false;
  if (c < b.C) {
    const Row r = read_row(b, c);
    if (!r.malformed) {
      const Pend pe = pend[c];
      uint64_t s = slot_of_id(r.id, reg.mask);
      for (uint64_t probe = 0; probe <= reg.mask; ++probe) {
        uint64_t k = reg.e[s].key;
        if (k == kEmptyId)
          k = atomicCAS((unsigned long long*)&reg.e[s].key, (unsigned long long)kEmptyId,
                        (unsigned long long)r.id);
        if (k == kEmptyId) {
          inserted = true;
          break;
        }
        s = (s + 1) & reg.mask;
      }
      // not inserted: unreachable, the host keeps the table at most half full
      if (inserted) {
        RegEntry& e = reg.e[s];
        e.state = kStAccepted | ((pe.kinds >> 8) == CLAIM_EV_OFFLOADED ? kStOffloaded : 0u);
        e.nblk = r.n;
        e.ntok = r.ntok;
        e.chain = pe.aux0;
        e.fpoff = store_at(fpo, fp_base, c, r.bo0);
        e.gen = gen;
        // leading_prefix_at_least(k): the blocks holding the first k tokens
        uint32_t pred = r.n;
        if (b.pred) {
          const uint64_t k = b.pred[c];
          const uint64_t kb = k / bs + (k % bs != 0);
          if (kb < r.n) pred = (uint32_t)kb;
        }
        e.pred = pred;
      }
    }
  }
  wave_count(&ctr->reg_count, inserted);
}

// ----------------------------------------------------------------- restore

// Registration pass 2: duplicate ownership, and each block's latest
// registration.  Every position an offloaded claim of the batch registered
// compares its block with the block stored for its identity; a different
// one makes the identity ambiguous (counted once, by the call that sets the
// flag).  It also raises the block's owner_at to its identity-store index
// + 1: store indices grow with the call, the claim and the position, so the
// maximum is the block's latest registration (k_holders then reads its
// identity).  Claims are taken in reverse batch order and owner_at is read
// before the atomic, so most positions find a later one already there and
// skip it.
template <int W>
__global__ void __launch_bounds__(kThreads) k_register_owners(BatchDev b, RegDev reg, IdDev ids,
                                                              uint32_t nb, uint32_t bs,
                                                              uint64_t fp_base,
                                                              const uint64_t* __restrict__ fpo,
                                                              uint64_t* __restrict__ owner_at,
                                                              Counters* __restrict__ ctr) {
  const uint64_t c_fwd = group_claim<W>();
  if (c_fwd >= b.C) return;
  const uint64_t c = b.C - 1 - c_fwd;
  const uint32_t gl = (threadIdx.x & 63) & (W - 1);
  const Row r = read_row(b, c);
  const uint64_t nt = (r.ntok + bs - 1) / bs;
  uint32_t missing = 0;
  for (uint64_t j = gl; j < r.n; j += W)
    if (b.bi[(uint64_t)r.bo0 + j] >= nb) missing = 1;
  missing = group_or<W>(missing);
  const bool offloaded = !r.malformed && r.n > 0 && !missing && (uint64_t)r.n == nt;
  if (!offloaded) return;
  const uint64_t at0 = store_at(fpo, fp_base, c, r.bo0);
  for (uint64_t j0 = 0; j0 < r.n; j0 += W) {
    const uint64_t j = j0 + gl;
    uint32_t amb = 0;
    if (j < r.n) {
      const uint64_t key = reg.idn[at0 + j];
      const uint32_t blk = b.bi[(uint64_t)r.bo0 + j];
      const unsigned long long mine = at0 + j + 1;
      const IdEntry* e = id_find(ids, key);
      if (e && e->block != blk &&
          !(atomicOr((uint32_t*)&e->flags, kIdAmbiguous) & kIdAmbiguous))
        amb = 1;
      if (*(volatile unsigned long long*)(owner_at + blk) < mine)
        atomicMax((unsigned long long*)(owner_at + blk), mine);
    }
    wave_count(&ctr->id_ambiguous, amb);
  }
}

// Registration pass 3: each block of the offload whose latest registration
// belongs to this call (owner_at past the call's first store index) now
// holds that registration's identity.
__global__ void __launch_bounds__(kThreads) k_holders(const uint32_t* __restrict__ uniq,
                                                      const Counters* __restrict__ ctr,
                                                      const uint64_t* __restrict__ owner_at,
                                                      const uint64_t* __restrict__ idn,
                                                      uint64_t fp_base,
                                                      uint64_t* __restrict__ holder) {
  const uint32_t U = ctr->uniq_count;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads;
  for (uint64_t u = (uint64_t)blockIdx.x * kThreads + threadIdx.x; u < U; u += stride) {
    const uint32_t b = uniq[u];
    const uint64_t o = owner_at[b];
    if (o > fp_base) holder[b] = idn[o - 1];
  }
}

__global__ void __launch_bounds__(kThreads) k_flips(uint32_t* __restrict__ pool32, uint32_t nb,
                                                    uint64_t chunk_bytes, uint32_t n,
                                                    const uint32_t* __restrict__ blocks,
                                                    const uint64_t* __restrict__ bits) {
  const uint32_t f = blockIdx.x * kThreads + threadIdx.x;
  if (f >= n) return;
  const uint64_t byte = bits[f] >> 3;
  const uint64_t p = byte / chunk_bytes, q = byte % chunk_bytes;
  const uint64_t addr = (p * nb + blocks[f]) * chunk_bytes + q;
  atomicXor(pool32 + (addr >> 2), 1u << ((addr & 3) * 8 + (bits[f] & 7)));
}

// Reported load failures: the block's latest failure takes the restore's
// generation (every claim that recorded the block at an earlier generation
// now fails there).
__global__ void __launch_bounds__(kThreads) k_set_failed(BlockRes* __restrict__ bres, uint32_t n,
                                                         const uint32_t* __restrict__ blocks,
                                                         uint64_t gen) {
  const uint32_t f = blockIdx.x * kThreads + threadIdx.x;
  if (f < n) bres[blocks[f]].fail_gen = gen;
}

// Copy staged blocks (those in the unique list) back into the pool.
__global__ void __launch_bounds__(kThreads) k_unstage(u32x4* __restrict__ pool, uint32_t nb,
                                                      uint32_t chunk_vecs, uint32_t planes,
                                                      const uint32_t* __restrict__ uniq,
                                                      const Counters* __restrict__ ctr,
                                                      const uint32_t* __restrict__ slot_of,
                                                      const u32x4* __restrict__ staging) {
  const uint64_t per_block = (uint64_t)planes * chunk_vecs;
  const uint64_t total = (uint64_t)ctr->uniq_count * per_block;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const uint64_t u = i / per_block, r = i % per_block;
    const uint32_t b = uniq[u];
    const uint64_t p = r / chunk_vecs, v = r % chunk_vecs;
    pool[(p * nb + b) * chunk_vecs + v] = staging[(uint64_t)slot_of[b] * per_block + r];
  }
}

__global__ void __launch_bounds__(kThreads) k_restore_claims(BatchDev b, RegDev reg,
                                                             uint32_t* __restrict__ cnt,
                                                             Pend* __restrict__ pend) {
  const uint64_t c = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
  if (c >= b.C) return;
  const Row r = read_row(b, c);
  cnt[c] = 0;
  if (r.malformed) return;
  const int64_t s = reg_find(reg, r.id);
  if (s < 0) return;
  const uint32_t state = reg.e[s].state;
  if (!(state & kStOffloaded)) return;
  // a plain store: every lane that finds this claim (a batch may present
  // it twice) stores the same value, and nothing else changes the state
  // while this kernel runs
  if (!(state & kStRestoreRequired)) reg.e[s].state = state | kStRestoreRequired;
  Pend pe;
  pe.aux0 = reg.e[s].nblk;
  pe.aux1 = 0;
  pe.kinds = CLAIM_EV_RESTORE_REQUIRED;
  pe.j = kNone;
  pe.phys = kNone;
  pe.pad = 0;
  pend[c] = pe;
  cnt[c] = 1;
}

// ------------------------------------------------------------------- check

struct CheckState {
  const BlockRes* bres;
};

template <int W>
__global__ void __launch_bounds__(kThreads) k_check(BatchDev b, RegDev reg, CheckState st,
                                                    uint32_t nb, uint32_t bs, uint64_t seed,
                                                    claim_outcome* __restrict__ out,
                                                    uint32_t* __restrict__ cnt,
                                                    Pend* __restrict__ pend) {
  __shared__ uint64_t tkey[kMaxBlockSize];
  load_token_keys(tkey, bs, seed);
  const uint64_t c = group_claim<W>();
  if (c >= b.C) return;
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t gl = lane & (W - 1), gbase = lane & ~(uint32_t)(W - 1);
  const Row r = read_row(b, c);
  const uint64_t nt = (r.ntok + bs - 1) / bs;
  const uint64_t n = r.n;

  uint32_t reasons = 0;
  uint64_t special = kNoKey;  // claim-level and length keys
  int64_t slot = -1;
  uint32_t na = 0, state = 0, pred = r.n;
  uint64_t acc_ntok = 0, acc_chain = 0, fpo = 0, q3 = kNoKey, acc_gen = 0;
  if (r.malformed) {
    reasons |= CLAIM_R_MALFORMED;
    special = kClaimLevelKey;
  } else {
    slot = reg_find(reg, r.id);
    if (slot < 0) {
      reasons |= CLAIM_R_NOT_ACCEPTED;
      special = kClaimLevelKey;
    } else {
      const RegEntry& e = reg.e[slot];
      state = e.state;
      na = e.nblk;
      pred = e.pred < r.n ? e.pred : r.n;
      acc_ntok = e.ntok;
      acc_chain = e.chain;
      fpo = e.fpoff;
      acc_gen = e.gen;
      if (!(state & kStOffloaded)) {
        reasons |= CLAIM_R_NOT_OFFLOADED;
        special = kClaimLevelKey;
      }
      if (!(state & kStRestoreRequired)) {
        reasons |= CLAIM_R_NO_RESTORE;
        special = kClaimLevelKey;
      }
      if (n != na) {
        reasons |= CLAIM_R_FOOTPRINT_MISMATCH;
        const uint64_t k = n < na ? n : na;
        special = k < special ? k : special;
      }
      if (acc_ntok != r.ntok) {  // the token counts part in this block
        reasons |= CLAIM_R_TOKEN_MISMATCH;
        q3 = (acc_ntok < r.ntok ? acc_ntok : r.ntok) / bs;
        special = q3 < special ? q3 : special;
      }
    }
    if (n == 0) {
      reasons |= CLAIM_R_EMPTY;
      special = kClaimLevelKey < special ? kClaimLevelKey : special;
    }
    if (n != nt) {
      reasons |= CLAIM_R_SHAPE_MISMATCH;
      const uint64_t k = n < nt ? n : nt;
      special = k < special ? k : special;
    }
  }
  const bool found = slot >= 0;
  const uint64_t common = n < na ? n : na;
  // the smallest length key (footprint length, block rows vs token blocks,
  // token counts): the only one of them that can decide, and whose h_j the
  // outcome may need
  uint64_t qmin = (found && n != na) ? common : kNoKey;
  if (!r.malformed && n != nt) qmin = (n < nt ? n : nt) < qmin ? (n < nt ? n : nt) : qmin;
  qmin = q3 < qmin ? q3 : qmin;
  // positions whose accepted identity is compared with the presented one
  uint64_t id_pos = 0;
  if (found) {
    const uint64_t acc_nt = (acc_ntok + bs - 1) / bs;
    id_pos = na < acc_nt ? na : acc_nt;
    id_pos = nt < id_pos ? nt : id_pos;
  }

  // Both chains start from the seed, and wherever the accepted h_{j-1}
  // equals the presented one, hh_j = splitmix64(acc_h_{j-1} ^ M_j) is the
  // presented h_j.  Each lane tests its position with hh_j against acc_h_j,
  // in parallel; by induction from j = 0, the first position q where they
  // differ is the first position where the two chains differ, the presented
  // h_j below it are the accepted ones, and hh_q is the presented h_q.  A
  // test past q may disagree with the serial chain's, but its key is larger
  // than q's and it lowers no minimum, so every output is the serial one.
  // A serial chain is walked only from p0 = min(q, id_pos) on, and only if
  // the outcome needs an h_j there.
  uint64_t best_pos = kNoKey;
  uint64_t q = kNoKey, h_qv = 0;  // first identity mismatch and the presented h there
  const uint64_t last = nt ? nt - 1 : kNoKey;
  // accepted h at the positions the outcome may report, taken from the
  // lanes that hold them (no loads after the loop)
  uint64_t acc_at_best = 0, acc_at_qmin = 0, acc_at_last = 0;
  uint64_t carry = seed;           // accepted h just before the window
  uint64_t intact = n < qmin ? n : qmin;  // first position with any problem (lane-local, then group min)
  const uint64_t L = n > nt ? n : nt;
  // Wide groups (long claims, many windows) load a window's position loads
  // and first token chunk during the previous window, so that a window
  // waits for one round trip (its block records) instead of two.
  constexpr bool kAhead = W >= 16;
  auto count_of = [&](uint64_t p) { return r.ntok - p * bs < bs ? r.ntok - p * bs : (uint64_t)bs; };
  uint32_t nx_blk = kNone, nx_acc_blk = kNone;
  uint64_t nx_acc_h = 0, nx_acc_d = 0;
  uint32_t nx_ch[kAhead ? 16 : 1];
  if constexpr (kAhead) {
    const uint64_t j = gl;
    if (j < n) nx_blk = b.bi[(uint64_t)r.bo0 + j];
    if (found && j < common) {
      nx_acc_blk = reg.fp[fpo + j];
      nx_acc_d = reg.dig[fpo + j];
    }
    if (j < id_pos) nx_acc_h = reg.idn[fpo + j];
    if (j < nt) prefetch_chunk(nx_ch, b.tok, r.to0 + j * bs, count_of(j));
  }
  for (uint64_t j0 = 0; j0 < L; j0 += W) {
    const uint64_t j = j0 + gl;
    // the window's loads that depend only on j, issued together
    uint32_t blk = kNone, acc_blk = kNone;
    uint64_t acc_h = 0, acc_d = 0;
    uint64_t m_sum = 0;
    if constexpr (kAhead) {
      blk = nx_blk;
      acc_blk = nx_acc_blk;
      acc_h = nx_acc_h;
      acc_d = nx_acc_d;
      if (j < nt) m_sum = multilinear_prefetched<1>(nx_ch, b.tok, r.to0 + j * bs, count_of(j), tkey);
    } else {
      if (j < n) blk = b.bi[(uint64_t)r.bo0 + j];
      if (found && j < common) {
        acc_blk = reg.fp[fpo + j];
        acc_d = reg.dig[fpo + j];
      }
      if (j < id_pos) acc_h = reg.idn[fpo + j];
      // the token loads go out first (they do not wait for blk)
      if (j < nt) m_sum = block_multilinear<1>(b.tok, r.to0 + j * bs, count_of(j), tkey);
    }
    // the block's record (restored digest, latest reported failure), loaded
    // unconditionally (block 0 stands in for a lane without a pool block)
    // so that it is in flight while the identity step runs; the empty asm
    // keeps every use, and so the wait, after it
    const uint32_t sb = (j < n && blk < nb) ? blk : 0u;
    u32x4 brec = *(const u32x4*)(st.bres + sb);
    if constexpr (kAhead) {  // the next window's loads, issued after the record's
      const uint64_t jn = j + W;
      nx_blk = jn < n ? b.bi[(uint64_t)r.bo0 + jn] : kNone;
      const bool has = found && jn < common;
      nx_acc_blk = has ? reg.fp[fpo + jn] : kNone;
      nx_acc_d = has ? reg.dig[fpo + jn] : 0;
      nx_acc_h = jn < id_pos ? reg.idn[fpo + jn] : 0;
      if (jn < nt) prefetch_chunk(nx_ch, b.tok, r.to0 + jn * bs, count_of(jn));
    }
    // the cache identity of block j, from the accepted h_{j-1}
    const uint64_t up = prev_lane64(acc_h);  // group lane gl-1's accepted identity
    const uint64_t hh = splitmix_step((gl == 0 ? carry : up) ^ m_sum);
    carry = group_read64<W>(acc_h, gbase, W - 1);
    asm volatile("" : "+v"(brec));
    const bool mism = j < id_pos && hh != acc_h;

    uint64_t my_key = kNoKey;
    if (j < n) {
      const bool own = found && j < common && blk == acc_blk;  // the claim recorded this block here
      if (found && j < common && blk != acc_blk) {
        reasons |= CLAIM_R_FOOTPRINT_MISMATCH;
        my_key = j;
      }
      if (blk >= nb) {
        reasons |= CLAIM_R_MISSING_ENTRY;
        my_key = j < my_key ? j : my_key;
      } else if (!found) {
        // a claim that was never accepted holds no offload record
      } else if (!own) {
        reasons |= CLAIM_R_NO_OFFLOAD_RECORD;
        my_key = j < my_key ? j : my_key;
      } else {
        // the claim's own record: a failure reported after its offload, or
        // a restored digest different from its own offload digest
        const uint64_t d_res = ((uint64_t)brec.y << 32) | brec.x;
        const uint64_t fail_gen = ((uint64_t)brec.w << 32) | brec.z;
        const bool lf = fail_gen > acc_gen;
        const bool mm = d_res != acc_d;
        if ((lf || mm) && j < intact) intact = j;
        if (j >= pred) {
          // past the predicate: the claimed prefix is still intact
          if (lf || mm) reasons |= CLAIM_R_BEYOND_PREDICATE;
        } else {
          if (lf) reasons |= CLAIM_R_LOAD_FAILED;
          if (mm) reasons |= CLAIM_R_DIGEST_MISMATCH;
          const uint64_t k = (1ull << 32) | j;
          if ((lf || mm) && k < my_key) my_key = k;
        }
      }
      if (my_key != kNoKey && j < intact) intact = j;
    }
    if (mism) {  // cache identity of block j
      reasons |= CLAIM_R_TOKEN_MISMATCH;
      my_key = j < my_key ? j : my_key;
      if (j < intact) intact = j;
    }
    if (q == kNoKey) {  // windows ascend: the first window with a mismatch holds q
      const uint32_t qi = group_first<W>(mism);
      if (qi < (uint32_t)W) {
        q = j0 + qi;
        h_qv = group_read64<W>(hh, gbase, qi);
      }
    }
    // the window's smallest key: positions ascend with the lane, so it is
    // the first lane's with a class-0 key, else the first lane's with any
    const uint64_t c0 = group_ballot<W>(my_key < (1ull << 32));
    const uint64_t c_any = group_ballot<W>(my_key != kNoKey);
    if (c_any) {
      const uint32_t li = (uint32_t)__builtin_ctzll(c0 ? c0 : c_any);
      const uint64_t rk = (c0 ? 0ull : (1ull << 32)) | (j0 + li);
      if (rk < best_pos) {
        best_pos = rk;
        acc_at_best = group_read64<W>(acc_h, gbase, li);
      }
    }
    if (qmin >= j0 && qmin < j0 + W) acc_at_qmin = group_read64<W>(acc_h, gbase, (uint32_t)(qmin - j0));
    if (last >= j0 && last < j0 + W) acc_at_last = group_read64<W>(acc_h, gbase, (uint32_t)(last - j0));
  }

  // the presented h at the positions the outcome reports: the winning key's
  // (if it has tokens) and the last token block's
  const uint64_t best_key = best_pos < special ? best_pos : special;
  const uint64_t js = best_key == kNoKey ? kNoKey : (best_key & 0xFFFFFFFFull);
  const bool want_js = js != kNone && js != kNoKey && js < nt;
  const uint64_t p0 = q < id_pos ? q : id_pos;  // presented h_j = accepted h_j below p0
  uint64_t h_js = 0, h_last = seed;
  bool tail = false;
  if (want_js) {
    // js is the winning position key's, or the smallest length key's (qmin)
    if (js < p0) h_js = best_key == best_pos ? acc_at_best : acc_at_qmin;
    else if (js == q) h_js = h_qv;
    else tail = true;
  }
  if (nt) {
    if (last < p0) h_last = acc_at_last;
    else if (last == q) h_last = h_qv;
    else tail = true;
  }
  if (tail) {  // serial chain from p0 (uncommon: a mismatch, or positions past the accepted ones)
    uint64_t h = p0 == 0 ? seed : reg.idn[fpo + p0 - 1];
    for (uint64_t j0 = p0; j0 < nt; j0 += W) {
      const uint64_t j = j0 + gl;
      uint64_t m_sum = 0;
      if (j < nt) {
        const uint64_t first = j * bs;
        const uint64_t count = r.ntok - first < bs ? r.ntok - first : bs;
        m_sum = block_multilinear<(W >= 16 ? 2 : 1)>(b.tok, r.to0 + first, count, tkey);
      }
      const uint64_t steps = nt - j0 < (uint64_t)W ? nt - j0 : (uint64_t)W;
      const uint64_t my_h = chain_window<W>(h, m_sum, gl, gbase, steps);
      if (want_js && js >= j0 && js < j0 + W && js != q && js >= p0)
        h_js = lane_read64(my_h, gbase + (uint32_t)(js - j0));
    }
    if (last >= p0 && last != q) h_last = h;
  }
  if (found && acc_chain != h_last) {  // whole-claim identity
    reasons |= CLAIM_R_TOKEN_MISMATCH;
    special = kClaimLevelKey < special ? kClaimLevelKey : special;
  }
  reasons = group_or<W>(reasons);
  intact = group_min64<W>(intact);
  if (gl != 0) return;

  const uint64_t best = best_pos < special ? best_pos : special;
  claim_outcome o;
  o.claim_id = r.id;
  o.num_blocks = r.n;
  o.reasons = reasons;
  o.intact_blocks = (uint32_t)intact;
  o.expected_digest = 0;
  o.observed_digest = 0;
  o.chain_hash = h_last;
  o.chain_hash_at_fail = 0;
  Pend pe;
  pe.pad = 0;
  pe.aux1 = 0;
  if (best == kNoKey) {
    o.code = CLAIM_MATERIALIZED;
    o.first_failing_block = kNone;
    o.phys_block = kNone;
    pe.kinds = CLAIM_EV_RESTORED;
    pe.aux0 = h_last;
    cnt[c] = 1;
  } else {
    const uint32_t cls = (uint32_t)(best >> 32);
    const uint32_t js = (uint32_t)(best & 0xFFFFFFFFull);
    o.code = cls == 0 ? CLAIM_UNKNOWN : CLAIM_RESTORE_FAILED_FAIL_CLOSED;
    o.first_failing_block = js;
    o.phys_block = (uint64_t)js < n ? b.bi[(uint64_t)r.bo0 + js] : kNone;
    if (cls == 1) {  // a class-1 key is always at a position the claim recorded
      o.expected_digest = reg.dig[fpo + js];
      o.observed_digest = st.bres[o.phys_block].d_res;
    }
    if (js != kNone && (uint64_t)js < nt) o.chain_hash_at_fail = h_js;
    if (cls == 1) {
      pe.kinds = CLAIM_EV_RESTORATION_FAILED | (CLAIM_EV_ACTIVE_REQUEST_REFUSED << 8);
      pe.aux0 = o.observed_digest;
      pe.aux1 = r.id;
      cnt[c] = 2;
    } else {
      pe.kinds = CLAIM_EV_OUTCOME_UNKNOWN;
      pe.aux0 = reasons;
      cnt[c] = 1;
    }
  }
  pe.j = o.first_failing_block;
  pe.phys = o.phys_block;
  out[c] = o;
  pend[c] = pe;
}

// ------------------------------------------------------------------ lookup

// A lookup probe issued ahead of its use: the whole 16-byte entry at the
// identity's home slot (key, block, flags), so that one load answers the
// common case; id_probe_resolve finishes it.
__device__ __forceinline__ u32x4 id_probe_issue(const IdDev& t, uint64_t key) {
  const IdEntry* e = key == 0 ? t.e + t.mask + 1 : t.e + slot_of_id(key, t.mask);
  return *(const u32x4*)e;
}

// The entry index of identity `key` (-1: not registered) from its home
// entry; when the home slot holds another identity the probe continues from
// the next slot (linear probing; the table is at most half full).
__device__ __forceinline__ int64_t id_probe_resolve(const IdDev& t, uint64_t key, u32x4 home) {
  const uint64_t k = ((uint64_t)home.y << 32) | home.x;
  if (key == 0) return (home.w & kIdUsed) ? (int64_t)(t.mask + 1) : -1;
  if (k == key) return (int64_t)slot_of_id(key, t.mask);
  if (k == 0) return -1;
  const IdEntry* e = id_find(t, key);
  return e ? (int64_t)(e - t.e) : -1;
}

// Reuse lookup: one group of W lanes per request; the group stops at the
// first token block whose identity is not a plain hit (absent, registered
// but ambiguous, or stale: its block was registered since under another
// identity, so it no longer holds this prefix; a stale identity stops the
// walk as an absent one does).
//
// Narrow groups (requests of a few blocks) hash one token block per lane,
// run the chain through the group and probe every lane's h_j.
//
// Wide groups (long requests) confirm positions without the serial chain.
// When h_j of the request is a registered identity, the claim that first
// registered it (IdSrc) has the same chain up to j and keeps its accepted
// identities acc_j, acc_{j+1}, ...  Lane i of a window computes
// hh = splitmix64(acc_{i-1} xor M_i) (h_prev for lane 0) and compares it
// with acc_i.  By induction from the window's start, below the first lane q
// whose hh differs (or that has no acc) the request's h equals acc, and at q
// it equals hh, so the window yields the request's h for lanes 0..q exactly,
// with no assumption about hash collisions.  Those lanes are probed in
// parallel; the first that is not a plain hit stops the lookup.  If none
// stops, a wholly confirmed window keeps the source, and otherwise lane q's
// own identity (a plain hit) gives the next source.  Without a source (the
// first position, or past the source claim's end) a window decides only its
// first position, which is the serial chain's step.  The outputs are the
// serial chain's.
template <int W>
__global__ void __launch_bounds__(kThreads) k_lookup(BatchDev b, IdDev ids,
                                                     const uint64_t* __restrict__ idn,
                                                     const uint64_t* __restrict__ holder,
                                                     uint32_t bs, uint64_t seed,
                                                     claim_lookup_result* __restrict__ out) {
  __shared__ uint64_t tkey[kMaxBlockSize];
  load_token_keys(tkey, bs, seed);
  const uint64_t c = group_claim<W>();
  if (c >= b.C) return;
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t gl = lane & (W - 1), gbase = lane & ~(uint32_t)(W - 1);
  const uint64_t id = b.ids[c];
  const uint64_t to0 = b.to[c], to1 = b.to[c + 1];
  const bool bad = id == kEmptyId || to0 > to1 || to1 > b.T;
  const uint64_t ntok = bad ? 0 : to1 - to0;
  const uint64_t nt = (ntok + bs - 1) / bs;

  uint64_t stop = kNoKey;  // (j << 1) | plain_miss of the first block that did not hit
  uint64_t h_at = seed;    // h_{hit - 1}
  if constexpr (W >= 16) {
    uint64_t j = 0, h_prev = seed;  // next position to decide, and h_{j-1}
    bool have_src = false;
    uint64_t a = 0, a_end = 0;  // idn[a] is the source's identity at position j
    // A window's first token chunk and accepted identity are loaded while
    // the previous window's probes are in flight (speculatively: as if that
    // window is confirmed whole; a window that is not discards them).
    auto count_of = [&](uint64_t p) { return ntok - p * bs < bs ? ntok - p * bs : (uint64_t)bs; };
    uint32_t ch[16];
    if ((uint64_t)gl < nt) prefetch_chunk(ch, b.tok, to0 + (uint64_t)gl * bs, count_of(gl));
    bool pre = true;        // ch holds the chunk of position j + gl
    uint64_t pre_acc = 0;   // idn[a + gl], when pre_has
    bool pre_has = false;
    while (j < nt) {
      const uint64_t jj = j + gl;
      uint64_t m_sum = 0;
      if (jj < nt) {
        const uint64_t first = to0 + jj * bs;
        m_sum = pre ? multilinear_prefetched<0>(ch, b.tok, first, count_of(jj), tkey)
                    : block_multilinear<0>(b.tok, first, count_of(jj), tkey);
      }
      const bool has_acc = have_src && jj < nt && a + gl < a_end;
      const uint64_t acc = has_acc ? (pre_has ? pre_acc : idn[a + gl]) : 0;
      const uint64_t up = prev_lane64(acc);  // group lane gl-1's acc
      const uint64_t hh = splitmix_step((gl == 0 ? h_prev : up) ^ m_sum);
      // first lane the source does not confirm (W: every lane up to nt)
      const uint32_t q = group_first<W>(!(jj >= nt || (has_acc && hh == acc)));
      const uint32_t known =
          q < (uint32_t)W ? q : (uint32_t)(nt - j < (uint64_t)W ? nt - j : (uint64_t)W) - 1;
      const uint64_t my_h = gl < q ? acc : hh;
      const bool probe = gl <= known;
      const u32x4 home = probe ? id_probe_issue(ids, my_h) : u32x4{0u, 0u, 0u, 0u};
      // the next window, if this one is confirmed whole
      const uint64_t jn = jj + W;
      pre = q == (uint32_t)W;
      pre_has = pre && have_src && jn < nt && a + W + gl < a_end;
      if (pre && jn < nt) prefetch_chunk(ch, b.tok, to0 + jn * bs, count_of(jn));
      if (pre_has) pre_acc = idn[a + W + gl];
      int64_t my_e = -1;
      bool amb = false, stale = false;
      if (probe) {
        my_e = id_probe_resolve(ids, my_h, home);
        const uint64_t home_slot = my_h == 0 ? ids.mask + 1 : slot_of_id(my_h, ids.mask);
        const bool at_home = (uint64_t)my_e == home_slot;
        amb = my_e >= 0 && ((at_home ? home.w : ids.e[my_e].flags) & kIdAmbiguous);
        if (my_e >= 0 && !amb) stale = holder[at_home ? home.z : ids.e[my_e].block] != my_h;
      }
      const uint64_t miss = group_ballot<W>(probe && (my_e < 0 || stale));
      const uint64_t stops = miss | group_ballot<W>(amb);
      if (stops) {  // the first position that is not a plain hit
        const uint32_t p = (uint32_t)__builtin_ctzll(stops);
        stop = ((j + p) << 1) | ((miss >> p) & 1u);
        h_at = p > 0 ? group_read64<W>(my_h, gbase, p - 1) : h_prev;
        break;
      }
      h_prev = group_read64<W>(my_h, gbase, known);
      if (q == (uint32_t)W) {
        a += known + 1;  // the whole window confirmed: keep following the source
      } else {
        const IdSrc src = ids.src[group_read64<W>((uint64_t)my_e, gbase, q)];
        have_src = true;
        a = src.at + 1;
        a_end = src.end;
      }
      j += known + 1;
    }
    if (stop == kNoKey) h_at = h_prev;
  } else {
    uint64_t h = seed;
    for (uint64_t j0 = 0; j0 < nt && stop == kNoKey; j0 += W) {
      const uint64_t j = j0 + gl;
      uint64_t m_sum = 0;
      if (j < nt) {
        const uint64_t first = j * bs;
        const uint64_t count = ntok - first < bs ? ntok - first : bs;
        m_sum = block_multilinear<0>(b.tok, to0 + first, count, tkey);
      }
      const uint64_t steps = nt - j0 < (uint64_t)W ? nt - j0 : (uint64_t)W;
      const uint64_t h_before = h;
      const uint64_t my_h = chain_window<W>(h, m_sum, gl, gbase, steps);
      uint64_t my_stop = kNoKey;
      if (j < nt) {
        const IdEntry* e = id_find(ids, my_h);
        if (!e)
          my_stop = (j << 1) | 1u;
        else if (e->flags & kIdAmbiguous)
          my_stop = j << 1;
        else if (holder[e->block] != my_h)
          my_stop = (j << 1) | 1u;  // stale: stops as an absent identity does
      }
      stop = group_min64<W>(my_stop);
      if (stop == kNoKey) {
        h_at = h;  // the whole window hit
      } else {
        const uint64_t js = stop >> 1;
        h_at = js > j0 ? lane_read64(my_h, gbase + (uint32_t)(js - 1 - j0)) : h_before;
      }
    }
  }
  if (gl != 0) return;

  claim_lookup_result o;
  o.request_id = id;
  o.reserved = 0;
  o.last_block = kNone;
  if (bad) {
    o.status = CLAIM_LOOKUP_UNKNOWN;
    o.hit_blocks = 0;
    o.hit_tokens = 0;
    o.chain_hash_at_hit = seed;
  } else {
    const uint64_t hit = stop == kNoKey ? nt : stop >> 1;
    const bool ambiguous = stop != kNoKey && !(stop & 1u);
    o.hit_blocks = (uint32_t)hit;
    o.hit_tokens = hit * bs < ntok ? hit * bs : ntok;
    o.chain_hash_at_hit = hit ? h_at : seed;
    if (hit) {
      const IdEntry* e = id_find(ids, h_at);
      o.last_block = e ? e->block : kNone;
    }
    o.status = ambiguous                ? CLAIM_LOOKUP_UNKNOWN
               : (hit == nt && hit > 0) ? CLAIM_LOOKUP_HIT
               : hit == 0               ? CLAIM_LOOKUP_MISS
                                        : CLAIM_LOOKUP_PARTIAL;
  }
  out[c] = o;
}

// ------------------------------------------------------------ event append

// Batches of up to kSmallEvents claims: one workgroup of 1024 threads
// appends the events and advances the log, in one launch.  It takes the
// claims in rounds of 1024, one per thread: coalesced loads of the counts,
// pending records and ids, a scan of the counts, the round's events built in
// LDS and copied to the log as contiguous 8-byte words.  (Four claims per
// thread with each thread storing its own events took 15.6 us for 4096
// claims.)
constexpr uint64_t kSmallEvents = 4096;

__global__ void __launch_bounds__(1024) k_events_small(const uint32_t* __restrict__ cnt,
                                                       const Pend* __restrict__ pend,
                                                       const uint64_t* __restrict__ ids, uint64_t C,
                                                       uint64_t ev_cap, Counters* __restrict__ ctr,
                                                       claim_event* __restrict__ log) {
  __shared__ uint32_t lds[17];
  __shared__ claim_event s_ev[2 * 1024];
  const uint64_t base_pos = ctr->log_count, base_seq = ctr->seq_next;
  // the call's events, counted first: all of them are appended, or none
  uint64_t all = 0;
  for (uint64_t c0 = 0; c0 < C; c0 += 1024) {
    const uint64_t c = c0 + threadIdx.x;
    uint32_t total;
    (void)block_exclusive_scan_1024(c < C ? cnt[c] : 0u, &total, lds);
    all += total;
  }
  if (base_pos + all > ev_cap) {
    if (threadIdx.x == 0) ctr->log_dropped = 1;
    return;  // uniform: every thread computed the same total
  }
  uint64_t run = 0;
  for (uint64_t c0 = 0; c0 < C; c0 += 1024) {
    const uint64_t c = c0 + threadIdx.x;
    const uint32_t v = c < C ? cnt[c] : 0u;
    Pend pe;
    uint64_t cid = 0;
    if (v) {
      pe = pend[c];
      cid = ids[c];
    }
    uint32_t total;
    uint32_t at = block_exclusive_scan_1024(v, &total, lds);  // also orders the LDS reuse
    for (uint32_t e = 0; e < v; ++e, ++at) {
      claim_event ev;
      ev.seq = base_seq + run + at;
      ev.claim_id = cid;
      ev.aux = e == 0 ? pe.aux0 : pe.aux1;
      ev.kind = (pe.kinds >> (8 * e)) & 0xFFu;
      ev.block_index = pe.j;
      ev.phys_block = pe.phys;
      ev.reserved = 0;
      s_ev[at] = ev;
    }
    __syncthreads();
    const uint64_t* src = (const uint64_t*)s_ev;
    uint64_t* dst = (uint64_t*)(log + base_pos + run);
    for (uint32_t i = threadIdx.x; i < total * (sizeof(claim_event) / 8); i += 1024) dst[i] = src[i];
    run += total;
    __syncthreads();  // s_ev is reused by the next round
  }
  if (threadIdx.x == 0) {
    ctr->log_count = base_pos + run;
    ctr->seq_next = base_seq + run;
  }
}

__global__ void __launch_bounds__(kThreads) k_tile_sums(const uint32_t* __restrict__ cnt,
                                                        uint64_t C, uint32_t* __restrict__ tsum) {
  __shared__ uint32_t lds[kThreads / 64];
  const uint64_t first = (uint64_t)blockIdx.x * kTile + threadIdx.x * (kTile / kThreads);
  uint32_t v = 0;
  for (int k = 0; k < kTile / kThreads; ++k)
    if (first + k < C) v += cnt[first + k];
  const uint32_t lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += lane_read(v, lane ^ o);
  if (lane == 0) lds[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) tsum[blockIdx.x] = lds[0] + lds[1] + lds[2] + lds[3];
}

// One workgroup: exclusive scan of the tile sums; reserves the call's range
// of the log.
__global__ void __launch_bounds__(1024) k_scan_tiles(uint32_t* __restrict__ tsum, uint64_t ntiles,
                                                     uint64_t ev_cap, Counters* __restrict__ ctr) {
  __shared__ uint32_t lds[17];
  __shared__ uint64_t run;
  if (threadIdx.x == 0) run = 0;
  __syncthreads();
  for (uint64_t t0 = 0; t0 < ntiles; t0 += 1024) {
    const uint64_t t = t0 + threadIdx.x;
    const uint32_t v = t < ntiles ? tsum[t] : 0;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan_1024(v, &total, lds);
    // tile prefixes can exceed 32 bits only for > 2^31 claims; kept 32-bit
    if (t < ntiles) tsum[t] = (uint32_t)(run + ex);
    __syncthreads();
    if (threadIdx.x == 0) run += total;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (ctr->log_count + run > ev_cap) {  // does not fit: the call's events are dropped
      ctr->call_pos = kDropped;
      ctr->log_dropped = 1;
    } else {
      ctr->call_pos = ctr->log_count;
      ctr->call_seq = ctr->seq_next;
      ctr->log_count += run;
      ctr->seq_next += run;
    }
  }
}

// Writes the events of one tile of kTile claims in rounds of 256 claims,
// one per thread: each round loads its claims' counts, pending records and
// ids with coalesced loads, scans the counts, builds the round's events in
// LDS and copies them to the log as contiguous 8-byte words (events are 40
// bytes, so a round's run of the log is 8-byte aligned).  Storing each
// event from its claim's thread instead puts consecutive stores 40 to 80
// bytes apart and costs about twice the time on a million-claim batch.
__global__ void __launch_bounds__(kThreads) k_write_events(const uint32_t* __restrict__ cnt,
                                                           const Pend* __restrict__ pend,
                                                           const uint64_t* __restrict__ ids,
                                                           uint64_t C,
                                                           const uint32_t* __restrict__ tprefix,
                                                           const Counters* __restrict__ ctr,
                                                           claim_event* __restrict__ log) {
  __shared__ uint32_t lds[kThreads / 64];
  __shared__ claim_event s_ev[2 * kThreads];
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t base_pos = ctr->call_pos, base_seq = ctr->call_seq;
  if (base_pos == kDropped) return;  // uniform: the call's events did not fit
  uint64_t run = tprefix[blockIdx.x];  // events of the tile before this round
  for (uint32_t r = 0; r < kTile / kThreads; ++r) {
    const uint64_t c = (uint64_t)blockIdx.x * kTile + r * kThreads + threadIdx.x;
    const uint32_t v = c < C ? cnt[c] : 0u;
    Pend pe;
    uint64_t cid = 0;
    if (v) {
      pe = pend[c];
      cid = ids[c];
    }
    // exclusive scan of the counts over the 256 threads
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t up = lane_read(incl, lane >= (uint32_t)o ? lane - o : lane);
      if (lane >= (uint32_t)o) incl += up;
    }
    if (lane == 63) lds[wave] = incl;
    __syncthreads();
    uint32_t before = 0, total = 0;
#pragma unroll
    for (uint32_t w = 0; w < kThreads / 64; ++w) {
      const uint32_t t = lds[w];
      before += w < wave ? t : 0u;
      total += t;
    }
    uint32_t at = before + incl - v;
    for (uint32_t e = 0; e < v; ++e, ++at) {
      claim_event ev;
      ev.seq = base_seq + run + at;
      ev.claim_id = cid;
      ev.aux = e == 0 ? pe.aux0 : pe.aux1;
      ev.kind = (pe.kinds >> (8 * e)) & 0xFFu;
      ev.block_index = pe.j;
      ev.phys_block = pe.phys;
      ev.reserved = 0;
      s_ev[at] = ev;
    }
    __syncthreads();
    const uint64_t* src = (const uint64_t*)s_ev;
    uint64_t* dst = (uint64_t*)(log + base_pos + run);
    for (uint32_t i = threadIdx.x; i < total * (sizeof(claim_event) / 8); i += kThreads)
      dst[i] = src[i];
    run += total;
    __syncthreads();  // s_ev and lds are reused by the next round
  }
}

// --------------------------------------------------------------- host side

const int kTimingSlots = 64;
const int kStages = 6;  // start, selected, digested, finalized, claims, events

// Fixed scratch of claim_check_static: per-claim event counts (4 B),
// pending events (32 B) and event-scan tile sums (4 B per 1024 claims) for
// batches of up to CLAIM_STATIC_MAX_CLAIMS claims, each part 256-byte
// aligned.
constexpr uint64_t kStaticCntOff = 0;
constexpr uint64_t kStaticPendOff =
    (kStaticCntOff + CLAIM_STATIC_MAX_CLAIMS * sizeof(uint32_t) + 255) / 256 * 256;
constexpr uint64_t kStaticTsumOff =
    (kStaticPendOff + CLAIM_STATIC_MAX_CLAIMS * sizeof(Pend) + 255) / 256 * 256;
constexpr uint64_t kStaticBytes =
    (kStaticTsumOff + (CLAIM_STATIC_MAX_CLAIMS + kTile - 1) / kTile * sizeof(uint32_t) + 255) / 256 * 256;

}  // namespace

// The scratch array itself: one copy on every GPU the library runs on, held
// until the process ends.  Host code never passes its name to a kernel (on
// the host it is only a stand-in for the symbol): claim_pool_create looks up
// its device address on each device once, with hipGetSymbolAddress, and
// claim_check_static hands that address to the kernels.
static __device__ __align__(256) uint8_t scratch[kStaticBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device

// The address of this device's scratch array (looked up on the first call
// for the device, which must be current).
int static_scratch(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return CLAIM_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return CLAIM_EHIP;
    }
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return CLAIM_OK;
}

}  // namespace

struct claim_pool {
  int device = 0;
  hipStream_t stream = nullptr;
  uint32_t flags = 0;
  uint32_t cus = 256;

  uint32_t planes = 0, bs = 0, nb = 0;
  uint64_t chunk_bytes = 0, chunk_vecs = 0, block_bytes = 0, seed = 0;
  KeyMap kmap{};  // key positions (head shards)
  void* kv = nullptr;

  int lpw = 32;
  uint32_t segs = 1, ps_total = 1, pgs = 1;
  uint32_t slots = 1;  // digest workgroups resident at once (per CU x CUs)

  uint64_t *d_off = nullptr, *partial = nullptr;
  BlockRes* bres = nullptr;  // per block: restored digest, latest reported failure
  uint8_t *valid_off = nullptr, *mark = nullptr;
  uint32_t *uniq = nullptr, *slot_of = nullptr;
  uint64_t* owner_at = nullptr;  // per block: identity-store index + 1 of its latest registration
  uint64_t* holder = nullptr;    // per block: the identity of that registration
  uint64_t gen = 0;              // generation of the latest offload or restore call

  uint64_t reg_mask = 0, max_claims = 0;
  RegEntry* reg = nullptr;
  uint32_t* fp_store = nullptr;
  uint64_t* idn_store = nullptr;  // accepted identities, parallel to fp_store
  uint64_t* dig_store = nullptr;  // each claim's own offload digests, parallel to fp_store
  uint64_t max_fp = 0, fp_used = 0;
  IdEntry* id_table = nullptr;
  IdSrc* id_src = nullptr;  // parallel to id_table
  uint64_t id_mask = 0;
  // staging of the current generation: the buffer staged offloads append
  // to, and the slots written to it so far
  const void* stage_base = nullptr;
  uint64_t stage_used = 0;
  uint64_t reg_used_ub = 0;  // upper bound on registered claims

  claim_event* log = nullptr;
  uint64_t ev_cap = 0, log_ub = 0;

  uint8_t* static_scratch = nullptr;  // this device's fixed scratch (claim_check_static)

  Counters* ctr = nullptr;
  Counters* host_ctr = nullptr;  // pinned

  uint64_t scratch_claims = 0, outcome_cap = 0;
  claim_outcome* outcomes = nullptr;
  uint32_t* cnt = nullptr;
  Pend* pend = nullptr;
  uint32_t* tsum = nullptr;
  uint64_t* fpo = nullptr;  // per-claim store offsets of a batch whose rows may share entries
  unsigned long long* dup_table = nullptr;
  uint64_t dup_cap = 0;
  uint64_t last_check_claims = 0;
  bool have_outcomes = false;

  uint32_t* f_blocks = nullptr;
  uint64_t* f_bits = nullptr;
  uint64_t f_cap = 0;

  hipEvent_t tev[kTimingSlots][kStages];
  bool tev_made = false;
  int t_head = 0, t_count = 0;  // ring of recorded checks not yet read
  claim_timing t_acc;
};

namespace {

int hip_status(hipError_t e) { return e == hipSuccess ? CLAIM_OK : CLAIM_EHIP; }

#define HIP_TRY(expr)                         \
  do {                                        \
    hipError_t e_ = (expr);                   \
    if (e_ != hipSuccess) return CLAIM_EHIP;  \
  } while (0)

#define TRY(expr)                \
  do {                           \
    int s_ = (expr);             \
    if (s_ != CLAIM_OK) return s_; \
  } while (0)

void dfree(void* p) {
  if (p) (void)hipFree(p);
}

template <typename T>
int dalloc(T** p, uint64_t count) {
  *p = nullptr;
  if (count == 0) count = 1;
  hipError_t e = hipMalloc((void**)p, count * sizeof(T));
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return CLAIM_ENOMEM;
  }
  return CLAIM_OK;
}

uint32_t grid_for(uint64_t threads, uint32_t cap = 1u << 20) {
  uint64_t g = (threads + kThreads - 1) / kThreads;
  if (g == 0) g = 1;
  return (uint32_t)(g < cap ? g : cap);
}

template <typename T>
int fill(claim_pool* P, T* p, uint64_t n, T v) {
  if (n == 0) return CLAIM_OK;
  hipLaunchKernelGGL(k_fill<T>, dim3(grid_for(n, 4096)), dim3(kThreads), 0, P->stream, p, n, v);
  return hip_status(hipGetLastError());
}

int fill_strided_u64(claim_pool* P, uint64_t* p, uint64_t n, uint32_t stride_words, uint64_t v) {
  if (n == 0) return CLAIM_OK;
  hipLaunchKernelGGL(k_fill_strided, dim3(grid_for(n, 4096)), dim3(kThreads), 0, P->stream, p, n,
                     stride_words, v);
  return hip_status(hipGetLastError());
}

uint64_t next_pow2(uint64_t x) {
  uint64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Group width for one claim per group: the mean row length, rounded up to a
// power of two in [2, 64].
int group_width(const claim_batch* b) {
  const uint64_t mean = b->num_claims ? (b->num_refs + b->num_claims - 1) / b->num_claims : 1;
  int w = 2;
  while (w < 64 && (uint64_t)w < mean) w <<= 1;
  return w;
}

BatchDev batch_dev(const claim_batch* b) {
  BatchDev d;
  d.C = b->num_claims;
  d.N = b->num_refs;
  d.T = b->num_tokens;
  d.ids = b->claim_ids;
  d.bo = b->block_offsets;
  d.bi = b->block_ids;
  d.to = b->token_offsets;
  d.tok = b->tokens;
  d.pred = b->predicate_tokens;
  return d;
}

RegDev reg_dev(claim_pool* P) {
  RegDev r;
  r.mask = P->reg_mask;
  r.e = P->reg;
  r.fp = P->fp_store;
  r.idn = P->idn_store;
  r.dig = P->dig_store;
  return r;
}

IdDev id_dev(claim_pool* P) {
  IdDev t;
  t.mask = P->id_mask;
  t.e = P->id_table;
  t.src = P->id_src;
  return t;
}

// Group width for a lookup batch: from the mean number of token blocks.
int lookup_group_width(const claim_batch* b, uint32_t bs) {
  const uint64_t per = b->num_claims ? (b->num_tokens + b->num_claims - 1) / b->num_claims : 1;
  const uint64_t mean = (per + bs - 1) / bs;
  int w = 2;
  while (w < 64 && (uint64_t)w < mean) w <<= 1;
  return w;
}

int check_batch(const claim_pool* P, const claim_batch* b) {
  if (!b || b->reserved != 0) return CLAIM_EINVAL;
  if (b->num_refs >= (uint64_t)kNone || b->num_claims > 0x7FFFFFFFu) return CLAIM_EINVAL;
  if (b->num_claims > 0 && (!b->claim_ids || !b->block_offsets || !b->token_offsets))
    return CLAIM_EINVAL;
  if (b->num_refs > 0 && !b->block_ids) return CLAIM_EINVAL;
  if (b->num_tokens > 0 && !b->tokens) return CLAIM_EINVAL;
  (void)P;
  return CLAIM_OK;
}

int ensure_claim_scratch(claim_pool* P, uint64_t C, bool for_check) {
  if (for_check && C > P->outcome_cap) {
    HIP_TRY(hipStreamSynchronize(P->stream));
    dfree(P->outcomes);
    P->outcomes = nullptr;
    P->outcome_cap = 0;
    P->have_outcomes = false;
    const uint64_t cap = C < 1024 ? 1024 : C;
    TRY(dalloc(&P->outcomes, cap));
    P->outcome_cap = cap;
  }
  if (C <= P->scratch_claims) return CLAIM_OK;
  HIP_TRY(hipStreamSynchronize(P->stream));
  dfree(P->cnt);
  dfree(P->pend);
  dfree(P->tsum);
  dfree(P->dup_table);
  dfree(P->fpo);
  P->cnt = nullptr;
  P->pend = nullptr;
  P->tsum = nullptr;
  P->dup_table = nullptr;
  P->fpo = nullptr;
  P->scratch_claims = 0;
  const uint64_t cap = C < 1024 ? 1024 : C;
  TRY(dalloc(&P->cnt, cap));
  TRY(dalloc(&P->pend, cap));
  TRY(dalloc(&P->tsum, (cap + kTile - 1) / kTile));
  TRY(dalloc(&P->fpo, cap + 1));
  P->dup_cap = next_pow2(2 * cap);
  TRY(dalloc(&P->dup_table, P->dup_cap));
  P->scratch_claims = cap;
  return CLAIM_OK;
}

// Mark + compact the blocks referenced by the batch into P->uniq.
int select_blocks(claim_pool* P, const claim_batch* b, int mode) {
  if (b->num_claims) {
    const BatchDev bd = batch_dev(b);
    const int W = group_width(b);
    const uint32_t grid = grid_for((uint64_t)b->num_claims * W, 0x7FFFFFFFu);
    switch (W) {
#define MARK_CASE(w)                                                                          \
  case w:                                                                                     \
    hipLaunchKernelGGL(k_mark<w>, dim3(grid), dim3(kThreads), 0, P->stream, bd, P->nb, mode, \
                       P->valid_off, P->slot_of, P->mark);                                    \
    break;
      MARK_CASE(2)
      MARK_CASE(4)
      MARK_CASE(8)
      MARK_CASE(16)
      MARK_CASE(32)
      MARK_CASE(64)
#undef MARK_CASE
      default:
        return CLAIM_EINVAL;
    }
    HIP_TRY(hipGetLastError());
  }
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, P->stream, P->mark, P->nb, P->uniq, P->ctr);
  return hip_status(hipGetLastError());
}

// The digest grid of one launch: pga piece groups read at a time, groups
// workgroups on each (grid = pga x groups).
struct DigestGrid {
  uint32_t pga, groups;
};

template <int LPW>
int launch_digest_lpw(claim_pool* P, DigestGrid gr, uint64_t* partial, void* staging,
                      int* wgs_per_cu) {
  const uint32_t cw = (uint32_t)(2 * P->chunk_vecs);
  const bool ragged = (uint64_t)P->segs * 64 * LPW != cw;
  const void* fn;
  if (ragged)
    fn = staging ? (const void*)k_digest<LPW, true, true> : (const void*)k_digest<LPW, true, false>;
  else
    fn = staging ? (const void*)k_digest<LPW, false, true> : (const void*)k_digest<LPW, false, false>;
  if (wgs_per_cu)  // occupancy query only
    return hip_status(hipOccupancyMaxActiveBlocksPerMultiprocessor(wgs_per_cu, fn, kThreads, 0));
  const u32x2* pool = (const u32x2*)P->kv;
  u32x2* st = (u32x2*)staging;
  const dim3 grid(gr.pga * gr.groups), block(kThreads);
#define GO(R, S)                                                                                \
  hipLaunchKernelGGL((k_digest<LPW, R, S>), grid, block, 0, P->stream, pool, P->nb, cw, P->planes, \
                     P->segs, gr.pga, gr.groups, P->uniq, P->ctr, P->seed, P->kmap, partial, st)
  if (ragged) {
    if (staging) GO(true, true); else GO(true, false);
  } else {
    if (staging) GO(false, true); else GO(false, false);
  }
#undef GO
  return hip_status(hipGetLastError());
}

// Launch the digest on grid gr (or, with wgs_per_cu, query its occupancy).
int launch_digest(claim_pool* P, DigestGrid gr, uint64_t* partial, void* staging,
                  int* wgs_per_cu = nullptr) {
  switch (P->lpw) {
#define DIGEST_CASE(l) \
  case l:              \
    return launch_digest_lpw<l>(P, gr, partial, staging, wgs_per_cu);
    DIGEST_CASE(1) DIGEST_CASE(2) DIGEST_CASE(4) DIGEST_CASE(8) DIGEST_CASE(12) DIGEST_CASE(16)
    DIGEST_CASE(24) DIGEST_CASE(32)
#undef DIGEST_CASE
    default:
      return CLAIM_EINVAL;
  }
}

int launch_finalize(claim_pool* P, DigestGrid gr, int mode, int staged, uint32_t slot0 = 0) {
  const uint32_t grid = grid_for((uint64_t)P->nb + gr.groups);  // slots <= U + groups
  hipLaunchKernelGGL(k_finalize, dim3(grid), dim3(kThreads), 0, P->stream, P->uniq, P->ctr,
                     P->partial, P->pgs, gr.groups, mode, staged, slot0, P->d_off, P->valid_off,
                     P->slot_of, P->bres);
  return hip_status(hipGetLastError());
}

// Per-claim scratch of one call: event counts, pending events, tile sums.
struct ClaimScratch {
  uint32_t* cnt;
  Pend* pend;
  uint32_t* tsum;
};

ClaimScratch pool_scratch(claim_pool* P) { return ClaimScratch{P->cnt, P->pend, P->tsum}; }

// Scan the per-claim event counts and append the events.
int append_events(claim_pool* P, const claim_batch* b, ClaimScratch sc) {
  const uint64_t C = b->num_claims;
  if (C == 0) return CLAIM_OK;
  if (C <= kSmallEvents) {
    hipLaunchKernelGGL(k_events_small, dim3(1), dim3(1024), 0, P->stream, sc.cnt, sc.pend,
                       b->claim_ids, C, P->ev_cap, P->ctr, P->log);
    return hip_status(hipGetLastError());
  }
  const uint64_t ntiles = (C + kTile - 1) / kTile;
  hipLaunchKernelGGL(k_tile_sums, dim3((uint32_t)ntiles), dim3(kThreads), 0, P->stream, sc.cnt, C,
                     sc.tsum);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(1024), 0, P->stream, sc.tsum, ntiles, P->ev_cap,
                     P->ctr);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(k_write_events, dim3((uint32_t)ntiles), dim3(kThreads), 0, P->stream, sc.cnt,
                     sc.pend, b->claim_ids, C, sc.tsum, P->ctr, P->log);
  return hip_status(hipGetLastError());
}

// Launch a claim-group kernel for the batch's group width.
#define LAUNCH_GROUPED(KERNEL, P, b, ...) LAUNCH_GROUPED_W(KERNEL, P, b, group_width(b), __VA_ARGS__)

#define LAUNCH_GROUPED_W(KERNEL, P, b, WIDTH, ...)                                              \
  do {                                                                                          \
    const int W_ = (WIDTH);                                                                     \
    const uint32_t grid_ = grid_for((uint64_t)(b)->num_claims * W_, 0x7FFFFFFFu);               \
    switch (W_) {                                                                               \
      case 2:                                                                                   \
        hipLaunchKernelGGL(KERNEL<2>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
      case 4:                                                                                   \
        hipLaunchKernelGGL(KERNEL<4>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
      case 8:                                                                                   \
        hipLaunchKernelGGL(KERNEL<8>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
      case 16:                                                                                  \
        hipLaunchKernelGGL(KERNEL<16>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
      case 32:                                                                                  \
        hipLaunchKernelGGL(KERNEL<32>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
      default:                                                                                  \
        hipLaunchKernelGGL(KERNEL<64>, dim3(grid_), dim3(kThreads), 0, (P)->stream, __VA_ARGS__); \
        break;                                                                                  \
    }                                                                                           \
    HIP_TRY(hipGetLastError());                                                                 \
  } while (0)

// Choose words per lane (LPW), segments per chunk and the digest grid.
// LPW is the largest instantiated width of at most kMaxExactLpw words (24,
// 16, 12, 8, ...) that divides the chunk's words-per-lane, so every segment
// is full and each wave streams up to 12 KiB per block; chunks that are not
// a whole number of 512-byte rows, or whose only exact widths are tiny, use
// the smallest width covering the chunk (at most 32) with a ragged last
// segment.  Measured on MI355X in one process over one allocation, two
// repetitions each: 16 words (8 KiB pieces, 32 KiB in flight per CU)
// instead of 32 (16 KiB pieces, 64 KiB) read the 8B pool 2.0 % faster
// (7.32 TB/s), the stress pool 2.6 %, 64 KiB chunks 1.8 %, fp8 and 64-plane
// 16 KiB pools 1.6-1.7 %, a 160-plane pool 0.8 %; the 70B pool 0.4 % and a
// 128-plane 16 KiB pool 2.3 % slower.  The 36 KiB MLA chunk keeps 24 words
// (12 words, 24 KiB in flight, read it 14 % slower).  The grid is
// persistent and fully resident (no tail of late waves): slots = workgroups
// per CU x CUs, shared by the piece groups read at a time (digest_grid).
// Workgroups per CU: enough for about
// kInflightPerCu bytes of loads in flight per CU (each wave keeps
// LPW x 512 bytes in flight), at most what can be resident.  Measured on
// MI355X in one process over one pool allocation, 32 KiB per CU read the
// pool faster than filling every resident slot: 8B 2.446 -> 2.394 ms,
// stress 4.340 -> 4.294, MLA 2.012 -> 1.972, the 70B head shard 2.046 ->
// 2.026 (2 per CU there), 70B unchanged (15.40 -> 15.43); more requests
// outstanding than the memory needs only queue.
constexpr int kInflightPerCu = 32 << 10;
constexpr int kMaxExactLpw = 24;

int choose_digest_shape(claim_pool* P) {
  static const int kLpw[] = {32, 24, 16, 12, 8, 4, 2, 1};  // instantiated widths, descending
  const uint64_t CW = 2 * P->chunk_vecs;  // 64-bit words per chunk
  const uint64_t Q = (CW + 63) / 64;      // words per lane to cover one chunk
  int best = 0;
  if (CW % 64 == 0)
    for (int d : kLpw)
      if (d <= kMaxExactLpw && Q % d == 0) {
        best = d;
        break;
      }
  if (best && best < 8 && Q > 32) best = 0;  // only tiny exact widths: use a ragged tail
  if (best == 0) {                           // ragged: the smallest width covering Q, at most 32
    best = 32;
    for (int d : kLpw)
      if ((uint64_t)d >= Q) best = d;
  }
  P->lpw = best;
  P->segs = (uint32_t)((Q + best - 1) / best);
  P->ps_total = P->planes * P->segs;
  P->pgs = (P->ps_total + 3) / 4;
  int per_cu = 0;
  TRY(launch_digest(P, DigestGrid{1, 1}, nullptr, nullptr, &per_cu));  // the kernel's occupancy
  const int wg_bytes = 4 * best * 64 * 8;  // loads in flight per workgroup
  const int want = kInflightPerCu / wg_bytes > 1 ? kInflightPerCu / wg_bytes : 1;
  if (per_cu > want) per_cu = want;
  if (per_cu < 1) per_cu = 1;
  P->slots = (uint32_t)per_cu * P->cus;
  return CLAIM_OK;
}

// How many piece groups a digest launch reads at a time (pga, a divisor of
// the piece-group count, so that every workgroup runs the same number of
// phases) and how many workgroups share each (groups = slots / pga).
//
// Reading every piece group at once suits pools of up to about 13 GB.
// From kTwoPhaseBytes to kOnePhaseBytes of referenced blocks a launch reads
// in two phases when the piece groups split evenly in two at a plane
// chunk's edge (an even count, half of whose pieces make whole chunks), so
// that no chunk is read partly in each phase; otherwise in one.  Past
// kOnePhaseBytes it reads in phases of at most kPhaseBytes.  Measured on
// MI355X with 8 KiB pieces, each comparison in one process over one
// allocation, in several processes: two phases read the 17 GB 8B pool
// 0.7-1.6 % faster than one (32 piece groups at a time instead of 64; more
// phases were slower), the 30 GB stress pool 0.4-0.8 % faster (14 instead
// of 28), 128-plane pools of 16 KiB chunks of 17 and 34 GB 1.8 % and 2.3 %
// faster, and 64-plane pools of 16 KiB chunks within 0.3 %.  MLA pools,
// whose 36 KiB chunks are three 12 KiB pieces so that half the piece groups
// end inside a chunk, read 1.1-1.5 % slower in two phases (13.5 and
// 17.1 GB), and the 13.1 GB 70B head shard no faster.
// Over the 105 GB 70B pool (160 piece groups), 2 piece groups at a time
// (phases of 1.3 GB) read 1.0-1.4 % faster than 5 (3.3 GB phases, the
// bound of 4 GiB used before), and every other size from 1 to 80 was slower
// than 2; an 84 GB pool read the same with 1 or 2 at a time.  With 16 KiB
// pieces, all piece groups at once read the 84 and 105 GB pools at only
// 6.77-6.84 TB/s against 7.07-7.10 in phases of 2.6-5.2 GB, while pools of
// 13 to 30 GB read at 6.96-7.20 TB/s in one phase.  That loss is not address
// translation (the phased launches took more translation misses: about
// 46 000 and 113 000 per launch against 2 000); the phased launches kept
// more requests outstanding at the memory interface (about 6 000-6 240 on
// average against 5 500-5 660).  A phase costs a key computation and a ring
// flush, which a pool with few blocks per workgroup feels (a 21 GB pool of
// 4000 blocks read in 80 phases: -6 %), so short phases start only past
// kOnePhaseBytes.  Independently, a launch whose one-phase grid would leave
// more than 15 % of the slots idle (many piece groups, few slots each)
// reads in phases that fill it (320 planes: 6.05 -> 7.2 TB/s).  A phase
// never has more piece groups than there are slots, so the grid stays one
// resident round.  refs bounds the launch's unique blocks.
constexpr uint64_t kTwoPhaseBytes = 14ull << 30;
constexpr uint64_t kOnePhaseBytes = 32ull << 30;
constexpr uint64_t kPhaseBytes = 3ull << 29;  // 1.5 GiB
constexpr uint32_t kMinFillPct = 85;

DigestGrid digest_grid(const claim_pool* P, uint64_t refs) {
  const uint64_t ub = std::max<uint64_t>(1, std::min<uint64_t>(refs, P->nb));
  const long double bytes = (long double)ub * P->block_bytes;
  DigestGrid best{1, 1};
  uint64_t best_fill = 0;
  const bool one = bytes <= (long double)kOnePhaseBytes;
  // two phases where half the piece groups end on a plane chunk's edge
  const bool two = one && bytes >= (long double)kTwoPhaseBytes && P->pgs % 2 == 0 &&
                   (2ull * P->pgs) % P->segs == 0;
  for (uint32_t d = P->pgs; d >= 1; --d) {
    if (P->pgs % d || d > P->slots) continue;  // a phase must fit the resident slots
    if (d > 1 && !one && bytes * d > (long double)kPhaseBytes * P->pgs) continue;
    if (two && 2 * d > P->pgs) continue;
    const uint64_t groups = std::min<uint64_t>(std::max<uint32_t>(1u, P->slots / d), ub);
    const uint64_t fill = (uint64_t)d * groups;
    if (fill * 100 >= (uint64_t)kMinFillPct * P->slots) return {d, (uint32_t)groups};
    if (fill > best_fill) {
      best_fill = fill;
      best = {d, (uint32_t)groups};
    }
  }
  return best;
}

void free_pool(claim_pool* P) {
  if (!P) return;
  void* ptrs[] = {P->d_off,    P->bres,      P->partial,  P->valid_off, P->mark,
                  P->uniq,     P->slot_of,   P->owner_at, P->holder,    P->reg,
                  P->fp_store, P->idn_store, P->dig_store, P->log,      P->ctr,
                  P->outcomes, P->cnt,       P->pend,     P->tsum,      P->dup_table,
                  P->f_blocks, P->f_bits,    P->id_table, P->id_src,    P->fpo};
  for (void* p : ptrs)
    if (p) dfree(p);
  if (P->host_ctr) (void)hipHostFree(P->host_ctr);
  if (P->tev_made)
    for (int i = 0; i < kTimingSlots; ++i)
      for (int s = 0; s < kStages; ++s) (void)hipEventDestroy(P->tev[i][s]);
  delete P;
}

int read_counters(claim_pool* P) {
  HIP_TRY(hipMemcpyAsync(P->host_ctr, P->ctr, sizeof(Counters), hipMemcpyDeviceToHost, P->stream));
  HIP_TRY(hipStreamSynchronize(P->stream));
  return CLAIM_OK;
}

// Fold the oldest recorded check's stage times into the accumulator.
int fold_timing_slot(claim_pool* P) {
  const int i = (P->t_head - P->t_count + kTimingSlots) % kTimingSlots;
  const bool stages = P->flags & CLAIM_POOL_STAGE_TIMING;
  HIP_TRY(hipEventSynchronize(P->tev[i][stages ? kStages - 1 : 2]));
  float ms[kStages - 1] = {0, 0, 0, 0, 0};
  for (int s = 0; s + 1 < kStages; ++s)
    if (stages || s == 1) HIP_TRY(hipEventElapsedTime(&ms[s], P->tev[i][s], P->tev[i][s + 1]));
  P->t_acc.calls += 1;
  P->t_acc.select_ms += ms[0];
  P->t_acc.digest_ms += ms[1];
  P->t_acc.finalize_ms += ms[2];
  P->t_acc.claims_ms += ms[3];
  P->t_acc.events_ms += ms[4];
  if (stages) P->t_acc.total_ms += ms[0] + ms[1] + ms[2] + ms[3] + ms[4];
  P->t_count -= 1;
  return CLAIM_OK;
}

// Stage events: 0 start, 1 selected, 2 digested, 3 finalized, 4 claims,
// 5 events.  Plain timing records only 1 and 2 (around the digest kernel).
int record_stage(claim_pool* P, int slot, int stage) {
  if (!(P->flags & CLAIM_POOL_TIMING)) return CLAIM_OK;
  if (!(P->flags & CLAIM_POOL_STAGE_TIMING) && stage != 1 && stage != 2) return CLAIM_OK;
  return hip_status(hipEventRecord(P->tev[slot][stage], P->stream));
}

}  // namespace

extern "C" {

const char* claim_strerror(int status) {
  switch (status) {
    case CLAIM_OK: return "ok";
    case CLAIM_EINVAL: return "invalid argument, layout or size";
    case CLAIM_ENOMEM: return "device allocation failed";
    case CLAIM_EHIP: return "HIP runtime error";
    case CLAIM_ENOSPC: return "capacity exceeded (registry, footprint, event log, staging or output)";
    case CLAIM_EDUP: return "duplicate claim id: acceptance refused";
    case CLAIM_ELIMIT: return "batch has more claims than claim_check_static's fixed scratch holds";
    default: return "unknown status";
  }
}

int claim_pool_create(const claim_pool_desc* d, claim_pool** out) {
  if (!d || !out) return CLAIM_EINVAL;
  *out = nullptr;
  if (d->num_layers == 0 || (d->planes_per_layer != 1 && d->planes_per_layer != 2) ||
      d->block_size == 0 || d->block_size > kMaxBlockSize || d->num_kv_heads == 0 ||
      d->head_dim == 0 || d->elem_bytes == 0 || d->num_blocks == 0 || d->num_blocks >= kNone ||
      !d->kv_base || ((uintptr_t)d->kv_base & 15) || d->max_claims == 0 ||
      d->event_capacity == 0 ||
      (d->flags & ~(CLAIM_POOL_TIMING | CLAIM_POOL_STAGE_TIMING)))
    return CLAIM_EINVAL;
  const uint64_t planes = (uint64_t)d->num_layers * d->planes_per_layer;
  const uint64_t chunk = (uint64_t)d->block_size * d->num_kv_heads * d->head_dim * d->elem_bytes;
  if (chunk % 16 || planes > 0xFFFFFFFFull || chunk / 16 > 0xFFFFFFFFull) return CLAIM_EINVAL;
  if (d->max_claims > (1ull << 40) || d->max_footprint > (1ull << 40)) return CLAIM_EINVAL;
  // a head shard: heads [first, first + num_kv_heads) of total_kv_heads,
  // each head's row a whole number of 64-bit words
  const uint32_t total_heads = d->total_kv_heads ? d->total_kv_heads : d->num_kv_heads;
  const uint64_t row_bytes = (uint64_t)d->head_dim * d->elem_bytes;
  if ((uint64_t)d->first_kv_head + d->num_kv_heads > total_heads) return CLAIM_EINVAL;
  if (total_heads != d->num_kv_heads && row_bytes % 8) return CLAIM_EINVAL;
  if ((uint64_t)d->block_size * total_heads * row_bytes / 8 > 0xFFFFFFFFull) return CLAIM_EINVAL;
  const long double need = (long double)planes * d->num_blocks * chunk;
  if (need > (long double)d->kv_bytes) return CLAIM_EINVAL;

  claim_pool* P = new (std::nothrow) claim_pool();
  if (!P) return CLAIM_ENOMEM;
  memset(&P->t_acc, 0, sizeof(P->t_acc));
  int rc = CLAIM_OK;
  do {
    if (hipGetDevice(&P->device) != hipSuccess) { rc = CLAIM_EHIP; break; }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, P->device) != hipSuccess) {
      rc = CLAIM_EHIP;
      break;
    }
    P->cus = cus > 0 ? (uint32_t)cus : 256;
    void* sp = nullptr;
    if ((rc = static_scratch(P->device, &sp))) break;
    P->static_scratch = (uint8_t*)sp;
    P->stream = (hipStream_t)d->stream;
    P->flags = d->flags;
    if (P->flags & CLAIM_POOL_STAGE_TIMING) P->flags |= CLAIM_POOL_TIMING;
    P->planes = (uint32_t)planes;
    P->bs = d->block_size;
    P->nb = d->num_blocks;
    P->chunk_bytes = chunk;
    P->chunk_vecs = chunk / 16;
    P->block_bytes = planes * chunk;
    P->seed = d->seed;
    P->kv = d->kv_base;
    P->kmap.chunk_words = (uint32_t)(chunk / 8);
    P->kmap.row_words = (uint32_t)(row_bytes / 8);
    P->kmap.heads = d->num_kv_heads;
    P->kmap.total = total_heads;
    P->kmap.first = d->first_kv_head;
    if ((rc = choose_digest_shape(P))) break;

    const uint64_t nb = d->num_blocks;
    if ((rc = dalloc(&P->d_off, nb)) || (rc = dalloc(&P->bres, nb)) ||
        (rc = dalloc(&P->partial, (uint64_t)P->pgs * (nb + P->slots))) ||
        (rc = dalloc(&P->valid_off, nb)) || (rc = dalloc(&P->mark, (nb + 15) / 16 * 16)) ||
        (rc = dalloc(&P->uniq, nb)) || (rc = dalloc(&P->slot_of, nb)) ||
        (rc = dalloc(&P->owner_at, nb)) || (rc = dalloc(&P->holder, nb)))
      break;
    P->max_claims = d->max_claims;
    const uint64_t cap = next_pow2(2 * d->max_claims);
    P->reg_mask = cap - 1;
    if ((rc = dalloc(&P->reg, cap))) break;
    P->max_fp = d->max_footprint;
    if ((rc = dalloc(&P->fp_store, d->max_footprint))) break;
    if ((rc = dalloc(&P->idn_store, d->max_footprint))) break;
    if ((rc = dalloc(&P->dig_store, d->max_footprint))) break;
    // every registered identity is a footprint position: at most half full
    const uint64_t id_cap = next_pow2(2 * d->max_footprint < 64 ? 64 : 2 * d->max_footprint);
    P->id_mask = id_cap - 1;
    if ((rc = dalloc(&P->id_table, id_cap + 1)) || (rc = dalloc(&P->id_src, id_cap + 1))) break;
    P->ev_cap = d->event_capacity;
    if ((rc = dalloc(&P->log, d->event_capacity))) break;
    if ((rc = dalloc(&P->ctr, 1))) break;
    if (hipHostMalloc((void**)&P->host_ctr, sizeof(Counters), hipHostMallocDefault) != hipSuccess) {
      P->host_ctr = nullptr;
      rc = CLAIM_ENOMEM;
      break;
    }
    if (P->flags & CLAIM_POOL_TIMING) {
      bool ok = true;
      for (int i = 0; i < kTimingSlots && ok; ++i)
        for (int s = 0; s < kStages && ok; ++s) ok = hipEventCreate(&P->tev[i][s]) == hipSuccess;
      if (!ok) { rc = CLAIM_EHIP; break; }
      P->tev_made = true;
    }
    if ((rc = fill<uint64_t>(P, P->d_off, nb, 0)) ||
        (rc = fill<uint64_t>(P, (uint64_t*)P->bres, 2 * nb, 0)) ||
        (rc = fill<uint8_t>(P, P->valid_off, nb, 0)) ||
        (rc = fill<uint64_t>(P, P->owner_at, nb, 0)) || (rc = fill<uint64_t>(P, P->holder, nb, 0)) ||
        (rc = fill<uint8_t>(P, P->mark, (nb + 15) / 16 * 16, 0)) || (rc = fill<uint32_t>(P, P->slot_of, nb, kNone)) ||
        (rc = fill<uint64_t>(P, (uint64_t*)P->reg, cap * (sizeof(RegEntry) / 8), 0)) ||
        (rc = fill_strided_u64(P, (uint64_t*)P->reg, cap, sizeof(RegEntry) / 8, kEmptyId)))
      break;
    // identity table: key 0 (empty), block kNone, flags 0
    if ((rc = fill<uint64_t>(P, (uint64_t*)P->id_table, 2 * (P->id_mask + 2), 0)) ||
        (rc = fill_strided_u64(P, (uint64_t*)P->id_table + 1, P->id_mask + 2, 2, (uint64_t)kNone)) ||
        (rc = fill<uint64_t>(P, (uint64_t*)P->id_src, 2 * (P->id_mask + 2), 0)))
      break;
    if ((rc = fill<uint64_t>(P, (uint64_t*)P->ctr, sizeof(Counters) / 8, 0))) break;
    if (hipStreamSynchronize(P->stream) != hipSuccess) { rc = CLAIM_EHIP; break; }
  } while (0);
  if (rc != CLAIM_OK) {
    free_pool(P);
    return rc;
  }
  *out = P;
  return CLAIM_OK;
}

int claim_pool_destroy(claim_pool* P) {
  if (!P) return CLAIM_OK;
  (void)hipSetDevice(P->device);
  hipError_t e = hipStreamSynchronize(P->stream);
  free_pool(P);
  return hip_status(e);
}

// Claims accepted ahead of the rest of a large batch.  Measured on MI355X
// over a batch of 10^6 claims of 1-4 blocks whose prefixes are shared
// (Zipf): acceptance 877-886 -> 807 us, the same with 16384; one inserting
// lane per distinct key in each wave instead measured the same, and both
// together no better.
constexpr uint64_t kAcceptFirst = 4096;

int claim_offload(claim_pool* P, const claim_batch* b, void* staging, uint64_t staging_bytes) {
  if (!P || ((uintptr_t)staging & 15)) return CLAIM_EINVAL;
  TRY(check_batch(P, b));
  HIP_TRY(hipSetDevice(P->device));
  const uint64_t C = b->num_claims;
  if (P->reg_used_ub + C > P->max_claims || P->log_ub + 2 * C > P->ev_cap) return CLAIM_ENOSPC;
  TRY(ensure_claim_scratch(P, C, false));

  // verdict: duplicates and the staged size, before any state changes
  TRY(fill<uint32_t>(P, &P->ctr->dup_flag, 1, 0u));
  const BatchDev bd = batch_dev(b);
  const RegDev rd = reg_dev(P);
  if (C) {
    TRY(fill<unsigned long long>(P, P->dup_table, P->dup_cap, (unsigned long long)kEmptyId));
    hipLaunchKernelGGL(k_dupcheck, dim3(grid_for(C, 0x7FFFFFFFu)), dim3(kThreads), 0, P->stream, bd,
                       rd, P->dup_table, P->dup_cap - 1, P->ctr);
    HIP_TRY(hipGetLastError());
  }
  TRY(select_blocks(P, b, kMarkAny));
  TRY(read_counters(P));
  if (P->host_ctr->dup_flag & kFlagDupId) return CLAIM_EDUP;
  const uint64_t U = P->host_ctr->uniq_count;
  // staging into the current generation's buffer appends after its slots;
  // any other buffer starts a new generation
  const bool append = staging && staging == P->stage_base;
  const uint64_t slot0 = append ? P->stage_used : 0;
  if (staging && (staging_bytes / P->block_bytes < slot0 + U || slot0 + U >= kNone))
    return CLAIM_ENOSPC;  // nothing changed
  // footprint and identity storage: the rows' own offsets when they are
  // disjoint (no row runs backwards), else a run per claim
  const uint64_t* fpo = nullptr;
  uint64_t fp_need = b->num_refs;
  if (P->host_ctr->dup_flag & kFlagBackwardRow) {
    hipLaunchKernelGGL(k_footprint_offsets, dim3(1), dim3(1024), 0, P->stream, bd, P->fp_used,
                       P->fpo);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(&fp_need, P->fpo + C, sizeof(uint64_t), hipMemcpyDeviceToHost,
                           P->stream));
    HIP_TRY(hipStreamSynchronize(P->stream));
    fpo = P->fpo;
  }
  if (P->fp_used + fp_need > P->max_fp) return CLAIM_ENOSPC;  // nothing changed

  // the offload digest of every block the batch references (staged from
  // slot slot0 of the current generation's buffer; another buffer starts a
  // new generation); acceptance then copies each claim's digests into its
  // own offload record
  P->gen += 1;
  if (staging && !append) TRY(fill<uint32_t>(P, P->slot_of, P->nb, kNone));
  const DigestGrid gr = digest_grid(P, b->num_refs);
  uint8_t* stage_at = staging ? (uint8_t*)staging + slot0 * P->block_bytes : nullptr;
  TRY(launch_digest(P, gr, P->partial, stage_at));
  TRY(launch_finalize(P, gr, 0, staging != nullptr, (uint32_t)slot0));
  if (C) {
    // A large batch's first claims are accepted in a launch of their own:
    // identities that many claims share (common prefixes) are then in the
    // table before the rest start, instead of every resident wave racing
    // to insert them into the same empty slots.
    const int W = group_width(b);
    const uint64_t first = C > 2 * kAcceptFirst ? kAcceptFirst : C;
    claim_batch part = *b;
    part.num_claims = (uint32_t)first;
    LAUNCH_GROUPED_W(k_accept, P, &part, W, bd, rd, id_dev(P), P->nb, P->bs, P->seed, P->fp_used,
                     fpo, P->d_off, P->fp_store, P->ctr, P->cnt, P->pend, 0ull, first);
    if (C > first) {
      part.num_claims = (uint32_t)(C - first);
      LAUNCH_GROUPED_W(k_accept, P, &part, W, bd, rd, id_dev(P), P->nb, P->bs, P->seed,
                       P->fp_used, fpo, P->d_off, P->fp_store, P->ctr, P->cnt, P->pend, first,
                       C);
    }
    hipLaunchKernelGGL(k_register_claims, dim3(grid_for(C, 0x7FFFFFFFu)), dim3(kThreads), 0,
                       P->stream, bd, rd, P->bs, P->fp_used, P->gen, fpo, P->pend, P->ctr);
    HIP_TRY(hipGetLastError());
    LAUNCH_GROUPED(k_register_owners, P, b, bd, rd, id_dev(P), P->nb, P->bs, P->fp_used, fpo,
                   P->owner_at, P->ctr);
    hipLaunchKernelGGL(k_holders, dim3(grid_for(U ? U : 1, 4096)), dim3(kThreads), 0, P->stream,
                       P->uniq, P->ctr, P->owner_at, P->idn_store, P->fp_used, P->holder);
    HIP_TRY(hipGetLastError());
    TRY(append_events(P, b, pool_scratch(P)));
  }
  TRY(read_counters(P));
  P->fp_used += fp_need;
  if (staging) {
    P->stage_base = staging;
    P->stage_used = slot0 + U;
  }
  P->reg_used_ub = P->host_ctr->reg_count;
  P->log_ub = P->host_ctr->log_count;
  return CLAIM_OK;
}

int claim_restore(claim_pool* P, const claim_batch* b, const void* staging,
                  uint64_t staging_bytes, const claim_fault_spec* f) {
  if (!P || ((uintptr_t)staging & 15)) return CLAIM_EINVAL;
  if (staging && staging_bytes / P->block_bytes < P->stage_used) return CLAIM_EINVAL;
  TRY(check_batch(P, b));
  HIP_TRY(hipSetDevice(P->device));
  const uint64_t C = b->num_claims;
  uint32_t nflip = 0, nfail = 0;
  if (f) {
    nflip = f->num_flips;
    nfail = f->num_load_failed;
    if ((nflip && (!f->flip_blocks || !f->flip_bits)) || (nfail && !f->load_failed_blocks))
      return CLAIM_EINVAL;
    for (uint32_t i = 0; i < nflip; ++i)
      if (f->flip_blocks[i] >= P->nb || f->flip_bits[i] >= 8 * P->block_bytes) return CLAIM_EINVAL;
    for (uint32_t i = 0; i < nfail; ++i)
      if (f->load_failed_blocks[i] >= P->nb) return CLAIM_EINVAL;
  }
  if (P->log_ub + C > P->ev_cap) return CLAIM_ENOSPC;
  TRY(ensure_claim_scratch(P, C, false));

  if (staging) {
    TRY(select_blocks(P, b, kMarkStaged));
    hipLaunchKernelGGL(k_unstage, dim3(grid_for((uint64_t)P->nb * P->planes * P->chunk_vecs, 65536)),
                       dim3(kThreads), 0, P->stream, (u32x4*)P->kv, P->nb, (uint32_t)P->chunk_vecs,
                       P->planes, P->uniq, P->ctr, P->slot_of, (const u32x4*)staging);
    HIP_TRY(hipGetLastError());
  }
  const uint64_t need = nflip > nfail ? nflip : nfail;
  if (need > P->f_cap) {
    HIP_TRY(hipStreamSynchronize(P->stream));
    dfree(P->f_blocks);
    dfree(P->f_bits);
    P->f_blocks = nullptr;
    P->f_bits = nullptr;
    P->f_cap = 0;
    TRY(dalloc(&P->f_blocks, need));
    TRY(dalloc(&P->f_bits, need));
    P->f_cap = need;
  }
  if (nflip) {
    HIP_TRY(hipMemcpyAsync(P->f_blocks, f->flip_blocks, nflip * sizeof(uint32_t),
                           hipMemcpyHostToDevice, P->stream));
    HIP_TRY(hipMemcpyAsync(P->f_bits, f->flip_bits, nflip * sizeof(uint64_t), hipMemcpyHostToDevice,
                           P->stream));
    hipLaunchKernelGGL(k_flips, dim3(grid_for(nflip)), dim3(kThreads), 0, P->stream,
                       (uint32_t*)P->kv, P->nb, P->chunk_bytes, nflip, P->f_blocks, P->f_bits);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipStreamSynchronize(P->stream));  // the fault lists may be reused next
  }
  P->gen += 1;
  if (nfail) {
    HIP_TRY(hipMemcpyAsync(P->f_blocks, f->load_failed_blocks, nfail * sizeof(uint32_t),
                           hipMemcpyHostToDevice, P->stream));
    hipLaunchKernelGGL(k_set_failed, dim3(grid_for(nfail)), dim3(kThreads), 0, P->stream, P->bres,
                       nfail, P->f_blocks, P->gen);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipStreamSynchronize(P->stream));
  }
  if (C) {
    hipLaunchKernelGGL(k_restore_claims, dim3(grid_for(C, 0x7FFFFFFFu)), dim3(kThreads), 0,
                       P->stream, batch_dev(b), reg_dev(P), P->cnt, P->pend);
    HIP_TRY(hipGetLastError());
    TRY(append_events(P, b, pool_scratch(P)));
  }
  P->log_ub += C;
  return CLAIM_OK;
}

}  // extern "C"

namespace {

// The check itself: outcomes to `out`, per-claim scratch in `sc`.
int check_body(claim_pool* P, const claim_batch* b, claim_outcome* out, ClaimScratch sc) {
  const uint64_t C = b->num_claims;
  int slot = 0;
  if (P->flags & CLAIM_POOL_TIMING) {
    if (P->t_count == kTimingSlots) TRY(fold_timing_slot(P));
    slot = P->t_head;
  }
  TRY(record_stage(P, slot, 0));
  TRY(select_blocks(P, b, kMarkOffloaded));  // recorded blocks of the well-formed rows
  TRY(record_stage(P, slot, 1));
  const DigestGrid gr = digest_grid(P, b->num_refs);
  TRY(launch_digest(P, gr, P->partial, nullptr));
  TRY(record_stage(P, slot, 2));
  TRY(launch_finalize(P, gr, 1, 0));
  TRY(record_stage(P, slot, 3));
  if (C) {
    CheckState st;
    st.bres = P->bres;
    LAUNCH_GROUPED(k_check, P, b, batch_dev(b), reg_dev(P), st, P->nb, P->bs, P->seed, out,
                   sc.cnt, sc.pend);
  }
  TRY(record_stage(P, slot, 4));
  TRY(append_events(P, b, sc));
  TRY(record_stage(P, slot, 5));
  if (P->flags & CLAIM_POOL_TIMING) {
    P->t_head = (P->t_head + 1) % kTimingSlots;
    P->t_count += 1;
  }
  P->log_ub += 2 * C;
  return CLAIM_OK;
}

}  // namespace

extern "C" {

int claim_check(claim_pool* P, const claim_batch* b) {
  if (!P) return CLAIM_EINVAL;
  TRY(check_batch(P, b));
  HIP_TRY(hipSetDevice(P->device));
  const uint64_t C = b->num_claims;
  if (P->log_ub + 2 * C > P->ev_cap) return CLAIM_ENOSPC;
  TRY(ensure_claim_scratch(P, C, true));
  TRY(check_body(P, b, P->outcomes, pool_scratch(P)));
  P->last_check_claims = C;
  P->have_outcomes = true;
  return CLAIM_OK;
}

int claim_check_static(claim_pool* P, const claim_batch* b, claim_outcome* out,
                       uint32_t out_cap) {
  if (!P) return CLAIM_EINVAL;
  TRY(check_batch(P, b));
  const uint64_t C = b->num_claims;
  if (C > CLAIM_STATIC_MAX_CLAIMS) return CLAIM_ELIMIT;
  if (C > 0 && !out) return CLAIM_EINVAL;
  if (out_cap < C || P->log_ub + 2 * C > P->ev_cap) return CLAIM_ENOSPC;
  HIP_TRY(hipSetDevice(P->device));
  uint8_t* sp = P->static_scratch;  // the device address, never the symbol's host name
  const ClaimScratch sc{(uint32_t*)(sp + kStaticCntOff), (Pend*)(sp + kStaticPendOff),
                        (uint32_t*)(sp + kStaticTsumOff)};
  TRY(check_body(P, b, out, sc));
  P->have_outcomes = false;  // this check's outcomes are in `out`
  return CLAIM_OK;
}

int claim_lookup(claim_pool* P, const claim_batch* b, claim_lookup_result* out,
                 uint32_t out_cap) {
  if (!P || !b || b->reserved != 0) return CLAIM_EINVAL;
  if (b->num_claims > 0x7FFFFFFFu) return CLAIM_EINVAL;
  if (b->num_claims > 0 && (!b->claim_ids || !b->token_offsets || !out)) return CLAIM_EINVAL;
  if (b->num_tokens > 0 && !b->tokens) return CLAIM_EINVAL;
  if (out_cap < b->num_claims) return CLAIM_ENOSPC;
  if (b->num_claims == 0) return CLAIM_OK;
  HIP_TRY(hipSetDevice(P->device));
  LAUNCH_GROUPED_W(k_lookup, P, b, lookup_group_width(b, P->bs), batch_dev(b), id_dev(P),
                   P->idn_store, P->holder, P->bs, P->seed, out);
  return CLAIM_OK;
}

int claim_identity_stats(claim_pool* P, uint64_t* entries, uint64_t* ambiguous) {
  if (!P) return CLAIM_EINVAL;
  HIP_TRY(hipSetDevice(P->device));
  TRY(read_counters(P));
  if (entries) *entries = P->host_ctr->id_entries;
  if (ambiguous) *ambiguous = P->host_ctr->id_ambiguous;
  return CLAIM_OK;
}

int claim_digest_grid(const claim_pool* P, uint64_t refs, claim_grid_info* out) {
  if (!P || !out) return CLAIM_EINVAL;
  const DigestGrid gr = digest_grid(P, refs);
  out->words_per_lane = (uint32_t)P->lpw;
  out->segments = P->segs;
  out->piece_groups = P->pgs;
  out->slots = P->slots;
  out->pga = gr.pga;
  out->groups = gr.groups;
  return CLAIM_OK;
}

int outcomes_read(claim_pool* P, claim_outcome* out, uint32_t out_cap, uint32_t* num_out,
                  claim_event* events, uint64_t ev_cap, uint64_t* num_events) {
  if (!P) return CLAIM_EINVAL;
  HIP_TRY(hipSetDevice(P->device));
  TRY(read_counters(P));
  const uint64_t nev = P->host_ctr->log_count;
  const uint64_t nout = P->have_outcomes ? P->last_check_claims : 0;
  const bool dropped = P->host_ctr->log_dropped != 0;
  if ((out && nout > out_cap) || (events && nev > ev_cap)) return CLAIM_ENOSPC;
  if (out) {
    if (nout) HIP_TRY(hipMemcpy(out, P->outcomes, nout * sizeof(claim_outcome), hipMemcpyDeviceToHost));
    if (num_out) *num_out = (uint32_t)nout;
  }
  if (events) {
    if (nev) HIP_TRY(hipMemcpy(events, P->log, nev * sizeof(claim_event), hipMemcpyDeviceToHost));
    if (num_events) *num_events = nev;
    P->host_ctr->log_count = 0;
    HIP_TRY(hipMemcpyAsync(&P->ctr->log_count, &P->host_ctr->log_count, sizeof(uint64_t),
                           hipMemcpyHostToDevice, P->stream));
    if (dropped) {
      P->host_ctr->log_dropped = 0;
      HIP_TRY(hipMemcpyAsync(&P->ctr->log_dropped, &P->host_ctr->log_dropped, sizeof(uint32_t),
                             hipMemcpyHostToDevice, P->stream));
    }
    HIP_TRY(hipStreamSynchronize(P->stream));
    P->log_ub = 0;
  } else {
    P->log_ub = nev;
  }
  return dropped ? CLAIM_ENOSPC : CLAIM_OK;
}

int claim_block_state_read(claim_pool* P, uint32_t first, uint32_t count, uint64_t* d_off,
                           uint64_t* d_res, uint8_t* valid_off, uint8_t* load_failed) {
  if (!P || (uint64_t)first + count > P->nb) return CLAIM_EINVAL;
  HIP_TRY(hipSetDevice(P->device));
  HIP_TRY(hipStreamSynchronize(P->stream));
  if (count == 0) return CLAIM_OK;
  if (d_off) HIP_TRY(hipMemcpy(d_off, P->d_off + first, count * 8ull, hipMemcpyDeviceToHost));
  if (valid_off) HIP_TRY(hipMemcpy(valid_off, P->valid_off + first, count, hipMemcpyDeviceToHost));
  // the per-block records (restored digest, failure generation) in one
  // contiguous copy, split on the host (a strided copy of 8-byte rows goes
  // row by row: about a minute for 4 M blocks)
  if (d_res || load_failed) {
    BlockRes* rec = new (std::nothrow) BlockRes[count];
    if (!rec) return CLAIM_ENOMEM;
    const hipError_t e =
        hipMemcpy(rec, P->bres + first, count * sizeof(BlockRes), hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      for (uint32_t i = 0; i < count; ++i) {
        if (d_res) d_res[i] = rec[i].d_res;
        if (load_failed) load_failed[i] = rec[i].fail_gen != 0;
      }
    delete[] rec;
    HIP_TRY(e);
  }
  return CLAIM_OK;
}

int claim_staging_reset(claim_pool* P) {
  if (!P) return CLAIM_EINVAL;
  HIP_TRY(hipSetDevice(P->device));
  TRY(fill<uint32_t>(P, P->slot_of, P->nb, kNone));  // queued: ordered with earlier restores
  P->stage_base = nullptr;
  P->stage_used = 0;
  return CLAIM_OK;
}

int claim_timing_read(claim_pool* P, claim_timing* out) {
  if (!P || !out || !(P->flags & CLAIM_POOL_TIMING)) return CLAIM_EINVAL;
  HIP_TRY(hipSetDevice(P->device));
  while (P->t_count > 0) TRY(fold_timing_slot(P));
  TRY(read_counters(P));
  *out = P->t_acc;
  out->last_unique = P->host_ctr->uniq_count;
  memset(&P->t_acc, 0, sizeof(P->t_acc));
  return CLAIM_OK;
}

}  // extern "C"
