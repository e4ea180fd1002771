/*
 * lifecycle.c -- the claim checker driven from plain C through its ABI alone:
 * device memory from hipMalloc, the default stream, no other runtime.  Used
 * by the GPU test of the C boundary (tests/test_gpu_c_abi.py), which writes
 * the input file, runs this program and compares what it writes with the
 * oracle.
 *
 *   lifecycle <input> <output>
 *
 * Input, little-endian: u32 layers, planes_per_layer, block_size, kv_heads,
 * head_dim, elem_bytes, num_blocks; u64 seed, pool_bytes; the pool's bytes;
 * u32 num_claims; u64 num_refs, num_tokens; u64 ids[C]; u32 block_offsets
 * [C+1]; u32 block_ids[N]; u64 token_offsets[C+1]; u32 tokens[T]; u32
 * num_flips, num_load_failed; u32 flip_blocks[F]; u64 flip_bits[F]; u32
 * load_failed[L].
 * Output: u32 status of each call (create, offload, restore, check, read);
 * u32 outcomes read, u64 events read; the outcomes (64 B each); the events
 * (40 B each).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "claimkv.h"

static void* read_n(FILE* f, size_t bytes) {
  void* p = malloc(bytes ? bytes : 1);
  if (!p || fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short input\n");
    exit(2);
  }
  return p;
}

static void* to_device(const void* host, size_t bytes) {
  void* d = NULL;
  if (hipMalloc(&d, bytes ? bytes : 16) != hipSuccess) {
    fprintf(stderr, "hipMalloc failed\n");
    exit(3);
  }
  if (bytes && hipMemcpy(d, host, bytes, hipMemcpyHostToDevice) != hipSuccess) {
    fprintf(stderr, "hipMemcpy failed\n");
    exit(3);
  }
  return d;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: lifecycle <input> <output>\n");
    return 2;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  uint32_t* geo = (uint32_t*)read_n(in, 7 * sizeof(uint32_t));
  uint64_t* sz = (uint64_t*)read_n(in, 2 * sizeof(uint64_t));
  void* pool_host = read_n(in, sz[1]);
  uint32_t C;
  uint64_t NT[2];
  if (fread(&C, 4, 1, in) != 1 || fread(NT, 8, 2, in) != 2) return 2;
  void* ids = read_n(in, 8ull * C);
  void* bo = read_n(in, 4ull * (C + 1));
  void* bi = read_n(in, 4ull * NT[0]);
  void* to = read_n(in, 8ull * (C + 1));
  void* tok = read_n(in, 4ull * NT[1]);
  uint32_t nf[2];
  if (fread(nf, 4, 2, in) != 2) return 2;
  uint32_t* flip_blocks = (uint32_t*)read_n(in, 4ull * nf[0]);
  uint64_t* flip_bits = (uint64_t*)read_n(in, 8ull * nf[0]);
  uint32_t* failed = (uint32_t*)read_n(in, 4ull * nf[1]);
  fclose(in);

  claim_pool_desc d;
  memset(&d, 0, sizeof(d));
  d.num_layers = geo[0];
  d.planes_per_layer = geo[1];
  d.block_size = geo[2];
  d.num_kv_heads = geo[3];
  d.head_dim = geo[4];
  d.elem_bytes = geo[5];
  d.num_blocks = geo[6];
  d.seed = sz[0];
  d.kv_base = to_device(pool_host, sz[1]);
  d.kv_bytes = sz[1];
  d.stream = NULL; /* the default stream */
  d.max_claims = 4ull * C + 16;
  d.max_footprint = 4ull * NT[0] + 16;
  d.event_capacity = 8ull * C + 16;

  claim_batch b;
  memset(&b, 0, sizeof(b));
  b.num_claims = C;
  b.num_refs = NT[0];
  b.num_tokens = NT[1];
  b.claim_ids = (const uint64_t*)to_device(ids, 8ull * C);
  b.block_offsets = (const uint32_t*)to_device(bo, 4ull * (C + 1));
  b.block_ids = (const uint32_t*)to_device(bi, 4ull * NT[0]);
  b.token_offsets = (const uint64_t*)to_device(to, 8ull * (C + 1));
  b.tokens = (const uint32_t*)to_device(tok, 4ull * NT[1]);

  claim_fault_spec f;
  f.num_flips = nf[0];
  f.num_load_failed = nf[1];
  f.flip_blocks = flip_blocks;
  f.flip_bits = flip_bits;
  f.load_failed_blocks = failed;

  int32_t st[5];
  claim_pool* pool = NULL;
  st[0] = claim_pool_create(&d, &pool);
  st[1] = pool ? claim_offload(pool, &b, NULL, 0) : -100;
  st[2] = pool ? claim_restore(pool, &b, NULL, 0, &f) : -100;
  /* the events of the offload and restore are read and dropped first */
  claim_event* ev = (claim_event*)malloc(sizeof(claim_event) * d.event_capacity);
  uint32_t n_out = 0;
  uint64_t n_ev = 0;
  if (pool && outcomes_read(pool, NULL, 0, NULL, ev, d.event_capacity, &n_ev) != CLAIM_OK) return 4;
  st[3] = pool ? claim_check(pool, &b) : -100;
  claim_outcome* out = (claim_outcome*)malloc(sizeof(claim_outcome) * (C ? C : 1));
  st[4] = pool ? outcomes_read(pool, out, C, &n_out, ev, d.event_capacity, &n_ev) : -100;
  if (pool) claim_pool_destroy(pool);

  FILE* o = fopen(argv[2], "wb");
  if (!o) return 2;
  fwrite(st, 4, 5, o);
  fwrite(&n_out, 4, 1, o);
  fwrite(&n_ev, 8, 1, o);
  fwrite(out, sizeof(claim_outcome), n_out, o);
  fwrite(ev, sizeof(claim_event), n_ev, o);
  fclose(o);
  printf("lifecycle: create %d offload %d restore %d check %d read %d: %u outcomes, %llu events (%s)\n",
         st[0], st[1], st[2], st[3], st[4], n_out, (unsigned long long)n_ev, claim_strerror(st[3]));
  hipFree(d.kv_base);
  hipFree((void*)b.claim_ids);
  hipFree((void*)b.block_offsets);
  hipFree((void*)b.block_ids);
  hipFree((void*)b.token_offsets);
  hipFree((void*)b.tokens);
  return 0;
}
