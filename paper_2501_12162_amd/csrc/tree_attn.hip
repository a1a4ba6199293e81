// Paged tree attention for batched tree verification on gfx950.
//
// Every node i of request r attends to the request's cached prefix (paged
// KV) followed by the nodes of its own root-to-node path, so one pass scores
// every candidate continuation of every draft token tree (section 2, draft
// token tree; section 4.3 step 4, verification of all trees in parallel).
//
// bf16 kernel, one workgroup (4 waves) per work unit (see plan.h):
//  * rows of a unit are (node, q-head-in-group) pairs of one kv-head, so the
//    G query heads that share a kv-head read each K/V byte once (GQA);
//  * K/V blocks of 32 keys go straight from HBM to LDS with 16-byte
//    global_load_lds (no staging registers) into a 5-stage ring: four
//    stages are in flight while one is multiplied, one barrier per block,
//    waits counted by hand (vmcnt) so the ring really overlaps; steps that
//    fetch whole prefix blocks run branch-free, five to a loop iteration,
//    so their LDS addresses are constants; when every request is one row
//    tile (no K/V byte is read twice) the loads carry the non-temporal hint;
//  * LDS rows are XOR-swizzled in 16-byte chunks so that both the K
//    fragment reads (16 keys x 16 B per quarter-wave) and the transposed V
//    reads (ds_read_b64_tr_b16) hit distinct banks;
//  * S^T = K Q^T and O^T = V^T P^T run on v_mfma_f32_16x16x32_bf16.  In this
//    orientation a lane owns one query row, so the online softmax needs no
//    cross-lane traffic except a max over the four 16-lane rows;
//  * the softmax folds the scale into one FMA per score (exp2 of
//    s*c - m*c) and only rescales a row's running state when its block max
//    rises more than 2^8 above the reference;
//  * the tree block (the request's own N_r nodes) is masked by 128-bit
//    ancestor sets built in LDS from parent[];
//  * prefixes longer than one chunk are split across workgroups; each writes
//    its partial (its own normalised output in bf16, reference max and
//    denominator in fp32) and a second, fully parallel kernel merges them
//    (the kernel boundary makes the partials of every XCD visible without
//    per-workgroup cache flushes).
#include <mutex>
#include <type_traits>

#include "accept_wave.h"
#include "adaserve.h"
#include "argmax_row.h"
#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace adaserve {

namespace {

constexpr int kThreads = 256;

// 16 bytes of zeros: the source of every DMA lane whose key is out of range,
// so no NaN from an unused page slot reaches LDS.  Its device address is
// passed in the kernel arguments (resolved once per device on the host).
__device__ __align__(16) uint32_t g_zero16[4];

typedef __attribute__((address_space(3))) char lds_char;

// LDS byte address of a __shared__ object (what M0 takes).
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const lds_char *)p;
}

// 16-byte loads from global memory straight into LDS (global_load_lds):
// lane l writes LDS bytes [lds + 16 l, +16).  Written as asm so that the
// compiler does not try to track these loads itself (it cannot follow a
// ring of stages across the loop and would wait for every load in flight
// before each LDS read); the "memory" clobber keeps every LDS access in
// program order around them, and the waits below are counted by hand.
// Setting M0 needs one wait state before the load that reads it.  The
// compiler reserves M0 and warns about the clobber; nothing else in this
// library uses M0 (LDS instructions on gfx950 do not read it).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// With NT the loads carry the non-temporal hint: used when every K/V byte of
// the launch is read by one workgroup only (single-tile requests), so the
// lines are not kept for a reuse that never comes (measured 3-6% faster on
// a 1 GB long-context batch, 6% slower where row tiles share a chunk).
template <bool NT>
__device__ __forceinline__ void dma16(const void *src, uint32_t lds) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :: "v"(src), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(src), "s"(lds) : "memory", "m0");
}
// Same with a wave-uniform base address and a 32-bit per-lane offset.
template <bool NT>
__device__ __forceinline__ void dma16_off(const void *base, uint32_t off, uint32_t lds) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
                 :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(N) with the other counters left open (for loads the
// compiler issued itself).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0xF70 | N);
}

// Waits until at most N of this wave's loads are in flight and its LDS
// operations are done, then the workgroup barrier.  No memory access moves
// across it.
template <int N>
__device__ __forceinline__ void wait_loads_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(N) : "memory");
}

// Index of the first plan entry whose unit_end (or group_end) exceeds `key`,
// or -1: every lane reads one entry per 64, so the whole table costs one
// round of loads instead of a chain of dependent ones.  Uniform result.
__device__ __forceinline__ int find_plan_entry(const TreeAttnArgs &a, int64_t key, bool groups) {
  static_assert(kPlanMax <= 3 * 64, "three rounds of 64 lanes cover the plan table");
  const int lane = threadIdx.x & 63;
  int32_t end[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int i = k * 64 + lane;
    end[k] = i < a.plan_count ? (groups ? a.plan[i].group_end : a.plan[i].unit_end) : INT32_MAX;
  }
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const unsigned long long hit = __ballot((int64_t)end[k] > key);
    if (hit) return k * 64 + __ffsll(hit) - 1;
  }
  return -1;
}

// Finds the request that owns logical index `idx`, counting either work units
// or (kv-head, row tile) groups per request.  Every lane of the wave ends with
// the same answer.  Returns false when idx is past the end.
__device__ bool locate_request(int64_t idx, bool count_groups, const TreeAttnArgs &a,
                               int32_t &r_out, int64_t &unit_base, int64_t &group_base) {
  const int lane = threadIdx.x & 63;
  int64_t cum_u = 0, cum_g = 0;
  for (int r0 = 0; r0 < a.num_requests; r0 += 64) {
    const int r = r0 + lane;
    int64_t nu = 0, ng = 0;
    if (r < a.num_requests) {
      int32_t n = a.node_indptr[r + 1] - a.node_indptr[r];
      n = min(max(n, 0), kMaxTreeNodes);
      const int32_t L = max(a.prefix_len[r], 0);
      ng = (int64_t)a.num_kv_heads * row_tiles(n, a.group, a.rows_per_tile);
      nu = ng * prefix_chunks(L, chunk_keys(n, a.group, a.rows_per_tile, a.chunk_target, a.chunk_floor));
    }
    const int64_t iu = wave_inclusive_scan(nu);
    const int64_t ig = wave_inclusive_scan(ng);
    const int64_t key = count_groups ? ig : iu;
    const int64_t base = count_groups ? cum_g : cum_u;
    const int64_t total = __shfl(key, 63, 64);
    if (idx < base + total) {
      const unsigned long long hit = __ballot(base + key > idx);
      const int first = __ffsll(hit) - 1;
      r_out = r0 + first;
      unit_base = cum_u + __shfl(iu - nu, first, 64);
      group_base = cum_g + __shfl(ig - ng, first, 64);
      return true;
    }
    cum_u += __shfl(iu, 63, 64);
    cum_g += __shfl(ig, 63, 64);
  }
  return false;
}

__device__ __forceinline__ uint32_t set_bit_in(uint32_t w, int word, int v) {
  return ((v >> 5) == word) ? (w | (1u << (v & 31))) : w;
}

// 16-byte chunk permutation of LDS row `row`: chunk c of the row is stored in
// slot c ^ swizzle(row).
template <int NCH>
__device__ __forceinline__ int swizzle(int row) {
  if (NCH == 16) return ((row & 7) << 1) | ((row >> 3) & 1);
  return (row >> 1) & 7;
}

template <int D, bool NT>
__global__ __launch_bounds__(kThreads, 2) void tree_attn_bf16_kernel(TreeAttnArgs a) {
  constexpr int KS = D / 32;                 // MFMA k-steps over the head dim
  constexpr int DT = D / 16;                 // 16-wide output tiles over the head dim
  constexpr int KB = kKeysPerBlock;          // 32 keys per pipeline stage
  constexpr int ROWB = D * 2;                // bytes per key row
  constexpr int NCH = D / 8;                 // 16-byte chunks per key row
  constexpr int BLK = KB * ROWB;             // bytes of K (or V) per block
  constexpr int WI = BLK / 1024 / 4;         // DMA wave-instructions per wave per tensor block
  constexpr int RPI = 1024 / ROWB;           // key rows covered by one wave-instruction
  constexpr float kRescaleLog2 = 8.f;

  // Scores run one block ahead of the PV product: step j multiplies K of
  // block j+1 and V of block j, and fetches K block j+5 and V block j+4.
  // Stage t of the five-stage ring holds [K block t+1 | V block t] (mod 5),
  // so a step reads one stage and refills another, and four of the five
  // stages are in flight while one is multiplied.  The ring is all the LDS
  // this kernel has (80 KB at D = 128, two workgroups per CU): page ids are
  // read from the block table with scalar loads, and the parents and
  // ancestor sets live in the V half of stage 4 until the first step
  // refills it (each lane keeps its own rows' ancestor sets in registers).
  constexpr int NST = 5;
  __shared__ __align__(1024) char ring[NST * 2 * BLK];
  int32_t *const par = (int32_t *)(ring + (NST - 1) * 2 * BLK + BLK);
  uint32_t *const anc = (uint32_t *)(ring + (NST - 1) * 2 * BLK + BLK + kMaxTreeNodes * 4);
  static_assert(kMaxTreeNodes * 4 * 5 <= BLK, "parents and ancestor sets fit in a V half-stage");

  if ((int64_t)blockIdx.x >= a.padded_grid) {
    // fused verification step: argmax workgroups follow the attention units,
    // taking CUs that no attention unit occupies
    const int64_t row = (int64_t)blockIdx.x - a.padded_grid;
    if (row < a.argmax_rows)
      argmax_row<true, kThreads>(a.logits, a.logit_stride, a.vocab, (int32_t)row, a.argmax_out, (float *)ring,
                                 (int *)(ring + 64));
    return;
  }
  const int64_t uid = xcd_swizzle(blockIdx.x, a.padded_grid);
  if (uid >= a.units) return;
  int32_t r, node_base, n, L, chunk_len;
  int64_t ubase;
  if (a.plan_count > 0) {
    // the dispatch-ordered plan in the kernel arguments
    const int lo = __builtin_amdgcn_readfirstlane(find_plan_entry(a, uid, false));
    if (lo < 0) return;
    r = plan_request(a.plan[lo].request_and_chunk);
    chunk_len = plan_chunk_keys(a.plan[lo].request_and_chunk);
    ubase = lo > 0 ? a.plan[lo - 1].unit_end : 0;
    node_base = a.plan[lo].node_base;
    n = plan_nodes(a.plan[lo].n_and_len);
    L = plan_prefix_len(a.plan[lo].n_and_len);
  } else {
    int64_t gbase;
    if (!locate_request(uid, false, a, r, ubase, gbase)) return;
    node_base = a.node_indptr[r];
    n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
    L = max(a.prefix_len[r], 0);
    chunk_len = chunk_keys(n, a.group, a.rows_per_tile, a.chunk_target, a.chunk_floor);
  }
  // Request values are uniform; make that visible so branches on them stay scalar.
  r = __builtin_amdgcn_readfirstlane(r);
  node_base = __builtin_amdgcn_readfirstlane(node_base);
  n = __builtin_amdgcn_readfirstlane(n);
  L = __builtin_amdgcn_readfirstlane(L);
  chunk_len = __builtin_amdgcn_readfirstlane(chunk_len);
  ubase = ((int64_t)__builtin_amdgcn_readfirstlane((int32_t)(ubase >> 32)) << 32) |
          (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)ubase);
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  // a chunk is whole 32-key blocks and its page ids fit the page-id registers
  if (chunk_len <= 0 || chunk_len > kMaxChunk || chunk_len % kKeysPerBlock != 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.group;
  const int RT = a.rows_per_tile;
  const int32_t tiles = row_tiles(n, G, RT);
  const int32_t chunks = prefix_chunks(L, chunk_len);
  const int64_t u = uid - ubase;
  const int32_t tile = (int32_t)(u % tiles);
  const int64_t rest = u / tiles;
  const int32_t g = (int32_t)(rest % a.num_kv_heads);
  const int32_t chunk = (int32_t)(rest / a.num_kv_heads);
  const int32_t M = n * G;
  const int32_t row0 = tile * RT;
  const int32_t row_end = min(M, row0 + RT);
  const bool last_chunk = chunk == chunks - 1;
  const int32_t k0 = chunk * chunk_len;
  const int32_t k1 = min(L, k0 + chunk_len);
  const int32_t n_prefix_blocks = k1 > k0 ? ceil_div(k1 - k0, KB) : 0;
  const int32_t n_full = k1 > k0 ? (k1 - k0) / KB : 0;   // prefix blocks that need no mask
  const int32_t n_tree_blocks = last_chunk ? ceil_div(n, KB) : 0;
  const int32_t nb = n_prefix_blocks + n_tree_blocks;
  const int32_t page0 = k0 / kPageSize;
  const int32_t npages = k1 > k0 ? ceil_div(k1, kPageSize) - page0 : 0;

  // ---- start-up: page ids, parents and queries, all loads in flight together.
  // The DMA rows of a wave lie in one 16-key page of each 32-key block (page
  // wave_page of the two); lane l of pgv[i] holds that page's id in prefix
  // block i*64 + l, or -1.
  const int wave_page = (wave * WI * RPI) / kPageSize;
  static_assert(kMaxChunk / KB <= 4 * 64, "page ids of a chunk fit in four lanes-wide registers");
  int32_t pgv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int32_t blk = i * 64 + lane;
    const int32_t e = page0 + blk * (KB / kPageSize) + wave_page;
    int32_t p = -1;
    if (blk < n_prefix_blocks && e < a.bt_stride) {
      p = a.block_table[(int64_t)r * a.bt_stride + e];
      if (p < 0 || p >= a.num_pages) p = -1;
    }
    pgv[i] = p;
  }
  (void)npages;
  if (last_chunk)
    for (int i = tid; i < n; i += kThreads) par[i] = a.parent[node_base + i];

  // Query fragments (B operand of S^T = K Q^T): lane holds row (lane & 15)
  // of each 16-row block, head-dim elements ks*32 + (lane >> 4)*8 .. +7.
  const int wrow0 = row0 + wave * 32;
  const bool wave_live = wrow0 < row_end;
  bf16x8 qf[2][KS];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = wrow0 + rb * 16 + (lane & 15);
    const bool valid = row < row_end;
    const int node = valid ? row / G : 0;
    const int hh = valid ? row - node * G : 0;
    const __bf16 *qp = (const __bf16 *)a.q +
                       ((int64_t)(node_base + node) * a.num_q_heads + g * G + hh) * D + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 v = {};
      if (valid) v = *(const bf16x8 *)(qp + ks * 32);
      qf[rb][ks] = v;
    }
  }
  // Let the start-up loads land before the first DMA, so the waits counted
  // by hand below only ever cover K/V blocks.
  wait_vmcnt<0>();

  // ---- DMA addressing: wave-instruction i of this wave fills LDS bytes
  // [(wave*WI + i)*1024, +1024) of a stage; lane `lane` lands on key row
  // dma_row[i], slot `slot`, so it fetches chunk slot ^ swizzle(row).  A
  // wave's rows lie in one 16-key page (wave_page of the two in a block), so
  // the page and its base address are wave-uniform; lanes add a 32-bit byte
  // offset inside the (page, kv-head) chunk or inside the tree block.
  const int slot = ((lane * 16) % ROWB) / 16;
  int dma_row[WI];
  uint32_t page_off[WI];   // bytes inside the (page, kv-head) chunk
  uint32_t tree_off[WI];   // bytes from the first key row of the tree block
  const int64_t tree_stride = (int64_t)a.num_kv_heads * D;   // elements between node rows
#pragma unroll
  for (int i = 0; i < WI; ++i) {
    dma_row[i] = (wave * WI + i) * RPI + (lane * 16) / ROWB;
    const int chunk_el = (slot ^ swizzle<NCH>(dma_row[i])) * 8;
    page_off[i] = (uint32_t)(((dma_row[i] % kPageSize) * D + chunk_el) * 2);
    tree_off[i] = (uint32_t)((dma_row[i] * tree_stride + chunk_el) * 2);
  }
  const int64_t page_stride_b = (int64_t)a.num_kv_heads * kPageSize * D * 2;   // bytes per page
  const int64_t head_off_b = (int64_t)g * kPageSize * D * 2;
  const int64_t tree_off_b = ((int64_t)node_base * a.num_kv_heads + g) * D * 2;
  // Fetches block blk of K (pool = k_pages, tree = k_tree) or of V into
  // `dst`.  Rows past the end of the block's keys, pages outside the pool and
  // blocks past the last one come from the zero line: every step issues the
  // same number of loads, so the waits below are constants.
  // `page` is this wave's physical page of block blk, or -1 (tree block,
  // entry past the block table row, or a page id outside the pool), read from
  // the page-id registers with lane reads (blk is uniform).
  auto page_of = [&](int blk) -> int32_t {
    if (blk >= n_prefix_blocks) return -1;
    const int l = blk & 63, hi = blk >> 6;
    const int32_t p0 = __builtin_amdgcn_readlane(pgv[0], l), p1 = __builtin_amdgcn_readlane(pgv[1], l);
    const int32_t p2 = __builtin_amdgcn_readlane(pgv[2], l), p3 = __builtin_amdgcn_readlane(pgv[3], l);
    return hi == 0 ? p0 : hi == 1 ? p1 : hi == 2 ? p2 : p3;
  };
  auto issue = [&](const void *pool, const void *tree, char *dst, int blk, int32_t page) {
    const char *base;
    int rows_left;
    const bool pre = blk < n_prefix_blocks;
    if (blk >= nb) {
      rows_left = 0;
      base = (const char *)tree;
    } else if (pre) {
      const int32_t p = __builtin_amdgcn_readfirstlane(page);
      rows_left = p >= 0 ? k1 - k0 - blk * KB : 0;
      base = (const char *)pool + head_off_b + (int64_t)max(p, 0) * page_stride_b;
    } else {
      const int tb = blk - n_prefix_blocks;
      rows_left = n - tb * KB;
      base = (const char *)tree + tree_off_b + (int64_t)tb * KB * tree_stride * 2;
    }
    const uint32_t lds = lds_addr(dst) + wave * WI * 1024;
    if (rows_left >= KB) {
#pragma unroll
      for (int i = 0; i < WI; ++i) dma16_off<NT>(base, pre ? page_off[i] : tree_off[i], lds + i * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < WI; ++i) {
        const bool ok = dma_row[i] < rows_left;
        dma16<NT>(ok ? (const void *)(base + (pre ? page_off[i] : tree_off[i])) : a.zero16, lds + i * 1024);
      }
    }
  };
  auto issue_k = [&](char *stage, int blk, int32_t page) { issue(a.k_pages, a.k_tree, stage, blk, page); };
  auto issue_v = [&](char *stage, int blk, int32_t page) {
    issue(a.v_pages, a.v_tree, stage + BLK, blk, page);
  };

  __syncthreads();  // par[] visible
  // Prologue issue order: K0 (stage 4), then (K1, V0), (K2, V1), (K3, V2),
  // (K4, V3) into stages 0 .. 3.
  int32_t pg4 = -1, pg5 = -1;   // pages of blocks j+4 and j+5 at step j
  if (nb > 0) {
    const int32_t pg0 = page_of(0), pg1 = page_of(1), pg2 = page_of(2), pg3 = page_of(3);
    pg4 = page_of(4);
    pg5 = page_of(5);
    issue_k(ring + 4 * 2 * BLK, 0, pg0);
    issue_k(ring + 0 * 2 * BLK, 1, pg1);
    issue_v(ring + 0 * 2 * BLK, 0, pg0);
    issue_k(ring + 1 * 2 * BLK, 2, pg2);
    issue_v(ring + 1 * 2 * BLK, 1, pg1);
    issue_k(ring + 2 * 2 * BLK, 3, pg3);
    issue_v(ring + 2 * 2 * BLK, 2, pg2);
    issue_k(ring + 3 * 2 * BLK, 4, pg4);
    issue_v(ring + 3 * 2 * BLK, 3, pg3);
  }

  // Ancestor sets (while the first blocks are in flight): bit j of node i's
  // set is 1 when j is on i's root-to-node path, i included.  The walk stops
  // at anything that is not a parent strictly before its child, so malformed
  // trees stay in bounds.
  if (last_chunk) {
    for (int i = tid; i < kMaxTreeNodes; i += kThreads) {
      uint32_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
      if (i < n) {
        int v = i;
        for (int step = 0; step < kMaxTreeNodes; ++step) {
          w0 = set_bit_in(w0, 0, v);
          w1 = set_bit_in(w1, 1, v);
          w2 = set_bit_in(w2, 2, v);
          w3 = set_bit_in(w3, 3, v);
          if (v == 0) break;
          const int p = par[v];
          if (p < 0 || p >= v) break;
          v = p;
        }
      }
      anc[i * 4 + 0] = w0;
      anc[i * 4 + 1] = w1;
      anc[i * 4 + 2] = w2;
      anc[i * 4 + 3] = w3;
    }
  }

  // Per-lane LDS offsets of the MFMA operand fragments inside a stage.
  const int q = lane >> 4, j16 = lane & 15;

  // The ancestor sets of this lane's two rows' nodes, in registers (named
  // scalars: an indexed array would be placed in scratch memory).
  uint32_t an00 = 0, an01 = 0, an02 = 0, an03 = 0, an10 = 0, an11 = 0, an12 = 0, an13 = 0;
  if (last_chunk) {
    __syncthreads();  // anc[] complete
    const int node0 = min((wrow0 + j16) / G, n - 1), node1 = min((wrow0 + 16 + j16) / G, n - 1);
    an00 = anc[node0 * 4 + 0], an01 = anc[node0 * 4 + 1], an02 = anc[node0 * 4 + 2], an03 = anc[node0 * 4 + 3];
    an10 = anc[node1 * 4 + 0], an11 = anc[node1 * 4 + 1], an12 = anc[node1 * 4 + 2], an13 = anc[node1 * 4 + 3];
  }
  int koff[KS];  // K fragment for keys kt*16 + j16 (add kt*16*ROWB), chunk ks*4 + q
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = j16 * ROWB + (((ks * 4 + q) ^ swizzle<NCH>(j16)) * 16);
  int voff[DT];  // transposed V read: key row q*4 + (j16 >> 2) (+16 for the upper half)
  {
    const int vrow = q * 4 + (j16 >> 2);
    const int sw = swizzle<NCH>(vrow);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      voff[dt] = vrow * ROWB + (((dt * 2 + ((j16 & 3) >> 1)) ^ sw) * 16) + (j16 & 1) * 8;
  }

  f32x4 o[2][DT];
  f32x4 osum[2];  // row sums of P, from an all-ones V tile on the matrix cores
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    osum[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[rb][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
  const float c = a.scale_log2;                      // raw score -> log2 units
  const float up_raw = kRescaleLog2 / c;             // rescale threshold in raw units
  float m_ref[2] = {-1e30f, -1e30f};                 // reference max of this lane's row (raw units)

  // S^T tiles of one block: s[rb][kt] holds keys kt*16 + q*4 + e of row j16.
  auto scores = [&](const char *kst, f32x4 (&s)[2][2]) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[0][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[1][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = *(const bf16x8 *)(kst + koff[ks] + kt * 16 * ROWB);
        s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[0][ks], s[0][kt], 0, 0, 0);
        s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[1][ks], s[1][kt], 0, 0, 0);
      }
    }
  };
  // Masks the partial prefix block and the tree blocks (ancestor sets).
  auto mask = [&](f32x4 (&s)[2][2], int blk) {
    {
      const bool tree_blk = blk >= n_prefix_blocks;
      const int tb = blk - n_prefix_blocks;
      const int valid = tree_blk ? min(KB, n - tb * KB) : min(KB, k1 - k0 - blk * KB);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        uint32_t aw = 0xffffffffu;
        if (tree_blk) {
          const uint32_t w0 = rb ? an10 : an00, w1 = rb ? an11 : an01;
          const uint32_t w2 = rb ? an12 : an02, w3 = rb ? an13 : an03;
          aw = (tb & 2) ? ((tb & 1) ? w3 : w2) : ((tb & 1) ? w1 : w0);
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = kt * 16 + q * 4 + e;
            const bool ok = key < valid && ((aw >> key) & 1u);
            s[rb][kt][e] = ok ? s[rb][kt][e] : -INFINITY;
          }
      }
    }
  };
  // Each row's block max.
  auto rowmax = [&](const f32x4 (&s)[2][2], float (&bm)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float m = __builtin_elementwise_maximum(
          __builtin_elementwise_maximum(s[rb][0][0], s[rb][0][1]), s[rb][0][2]);
      m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, s[rb][0][3]), s[rb][1][0]);
      m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, s[rb][1][1]),
                                        __builtin_elementwise_maximum(s[rb][1][2], s[rb][1][3]));
      bm[rb] = max_over_lane_rows(m);
    }
  };
  // Raises the reference max of the rows whose block max went more than
  // 2^8 above it, rescaling their running numerator and denominator.
  auto rescale = [&](const float (&bm)[2]) {
    const bool up0 = bm[0] > m_ref[0] + up_raw;
    const bool up1 = bm[1] > m_ref[1] + up_raw;
    if (__any(up0 || up1)) {
      const float n0 = up0 ? bm[0] : m_ref[0];
      const float n1 = up1 ? bm[1] : m_ref[1];
      const float a0 = up0 ? __builtin_amdgcn_exp2f((m_ref[0] - n0) * c) : 1.f;
      const float a1 = up1 ? __builtin_amdgcn_exp2f((m_ref[1] - n1) * c) : 1.f;
      m_ref[0] = n0;
      m_ref[1] = n1;
      osum[0] *= a0;
      osum[1] *= a1;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        o[0][dt] *= a0;
        o[1][dt] *= a1;
      }
    }
  };
  // P = 2^(s c - m c) in bf16, packed as the B operand of the PV product:
  // k-slot (q, e) is key q*4 + e (e < 4) or 16 + q*4 + (e - 4).
  auto probs = [&](const f32x4 (&s)[2][2], bf16x8 (&pk)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const float mc = m_ref[rb] * c;
      u32x4 w;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][kt][0], c, -mc));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][kt][1], c, -mc));
        const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][kt][2], c, -mc));
        const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][kt][3], c, -mc));
        w[kt * 2 + 0] = pack_bf16x2(p0, p1);
        w[kt * 2 + 1] = pack_bf16x2(p2, p3);
      }
      pk[rb] = __builtin_bit_cast(bf16x8, w);
    }
  };
  // O^T += V^T P^T and the row sums.  The transposed read hands lane
  // (q, j16) V[kbase + e][dt*16 + j16], e < 4.
  auto pv = [&](const char *vst, const bf16x8 (&pk)[2]) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vst + voff[dt]));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vst + voff[dt] + 16 * ROWB));
      const bf16x8 vf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[0], o[0][dt], 0, 0, 0);
      o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[1], o[1][dt], 0, 0, 0);
    }
    osum[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pk[0], osum[0], 0, 0, 0);
    osum[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pk[1], osum[1], 0, 0, 0);
  };

  f32x4 s[2][2];   // scores of the block whose PV product comes next
  float bm[2];     // their row maxima
  // Prologue: wait for K0 (the eight later prologue loads may still fly),
  // then the scores of block 0.
  if (nb > 0) {
    wait_loads_barrier<8 * WI>();
    if (wave_live) {
      scores(ring + 4 * 2 * BLK, s);
      if (n_full == 0) mask(s, 0);
      rowmax(s, bm);
    }
  }

  // Step j (its stage is cs = j mod 5): wait until K block j+1 and V block j
  // have landed (the loads of the three following steps may still fly),
  // barrier (every wave is done with K block j and V block j-1, whose stage
  // is refilled now), fetch K block j+5 and V block j+4, then P of block j,
  // scores of block j+1 and the PV product of block j; the scores of block
  // j+1 are masked (when they need it) and reduced last, while the PV
  // products run on the matrix cores.
  // `issue` for a block known to be a whole prefix block: no block-kind or
  // row-count branches, and a page outside the pool sends every lane to the
  // zero line (base = zero line, offset 0) without a branch.  Steps whose two
  // fetches are such blocks (most of a long chunk) take this form; it cuts
  // the scalar work of a step by about a third.
  auto issue_full = [&](const void *pool, char *dst, int32_t page) {
    const int32_t p = __builtin_amdgcn_readfirstlane(page);
    const uint32_t lds = lds_addr(dst) + wave * WI * 1024;
    const bool ok = p >= 0;
    const char *base = ok ? (const char *)pool + head_off_b + (int64_t)p * page_stride_b : (const char *)a.zero16;
#pragma unroll
    for (int i = 0; i < WI; ++i) dma16_off<NT>(base, ok ? page_off[i] : 0u, lds + i * 1024);
  };
  auto step = [&](int j, int cs, auto masked, auto has_next, auto full_fetch) {
    constexpr bool kMasked = decltype(masked)::value;
    constexpr bool kNext = decltype(has_next)::value;
    constexpr bool kFull = decltype(full_fetch)::value;
    const char *cur = ring + cs * (2 * BLK);
    if constexpr (kNext) {
      wait_loads_barrier<6 * WI>();
      char *fill = ring + (cs == 0 ? NST - 1 : cs - 1) * (2 * BLK);
      if constexpr (kFull) {
        issue_full(a.k_pages, fill, pg5);
        issue_full(a.v_pages, fill + BLK, pg4);
      } else {
        issue_k(fill, j + 5, pg5);
        issue_v(fill, j + 4, pg4);
      }
      pg4 = pg5;
      pg5 = page_of(j + 6);
    } else {
      wait_loads_barrier<0>();  // also drains the zero-line loads past the last block
    }
    if (wave_live) {
      rescale(bm);
      bf16x8 pk[2];
      probs(s, pk);
      if constexpr (kNext) {
        f32x4 sn[2][2];
        scores(cur, sn);
        pv(cur + BLK, pk);
        if constexpr (kMasked) mask(sn, j + 1);
        rowmax(sn, bm);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          s[rb][0] = sn[rb][0];
          s[rb][1] = sn[rb][1];
        }
      } else {
        pv(cur + BLK, pk);
      }
    }
  };
  using Yes = std::true_type;
  using No = std::false_type;
  int j = 0, cs = 0;
  auto next_stage = [](int c) { return c == NST - 1 ? 0 : c + 1; };
  // Blocks j+4 and j+5 whole prefix blocks: five steps per iteration (one
  // per ring stage, starting at stage 0), so every LDS address of a step is
  // a constant and folds into the instruction's offset.
  for (; j + 9 < n_full; j += 5) {
    step(j, 0, No{}, Yes{}, Yes{});
    step(j + 1, 1, No{}, Yes{}, Yes{});
    step(j + 2, 2, No{}, Yes{}, Yes{});
    step(j + 3, 3, No{}, Yes{}, Yes{});
    step(j + 4, 4, No{}, Yes{}, Yes{});
  }
  for (; j + 5 < n_full; ++j, cs = next_stage(cs)) step(j, cs, No{}, Yes{}, Yes{});
  for (; j + 1 < n_full; ++j, cs = next_stage(cs)) step(j, cs, No{}, Yes{}, No{});  // block j+1: full prefix block
  for (; j + 1 < nb; ++j, cs = next_stage(cs)) step(j, cs, Yes{}, Yes{}, No{});     // block j+1 needs the mask
  if (nb > 0) step(nb - 1, cs, No{}, No{}, No{});

  const int q4 = q * 4;
  const float l_tot[2] = {osum[0][0], osum[1][0]};
  if (chunks == 1) {
    if (!wave_live) return;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = wrow0 + rb * 16 + j16;
      if (row >= row_end) continue;
      const float inv = l_tot[rb] > 0.f ? 1.f / l_tot[rb] : 0.f;
      const int node = row / G, hh = row - (row / G) * G;
      __bf16 *op = (__bf16 *)a.out + ((int64_t)(node_base + node) * a.num_q_heads + g * G + hh) * D + q4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        u32x2 w;
        w[0] = pack_bf16x2(o[rb][dt][0] * inv, o[rb][dt][1] * inv);
        w[1] = pack_bf16x2(o[rb][dt][2] * inv, o[rb][dt][3] * inv);
        *(u32x2 *)(op + dt * 16) = w;
      }
    }
    return;
  }

  // ---- split prefix: write this chunk's partial: its own normalised output
  // in bf16 (a weighted mean of V rows, so bf16 keeps 2^-9 relative
  // precision), and its reference max and denominator in fp32;
  // tree_attn_combine_kernel merges the chunks after this kernel.
  if (!wave_live) return;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = wrow0 + rb * 16 + j16;
    if (row >= row_end) continue;
    const int64_t slot = uid * kMaxRowsPerTile + (row - row0);
    const float inv = l_tot[rb] > 0.f ? 1.f / l_tot[rb] : 0.f;
    __bf16 *wo = a.ws_o + slot * D + q4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      u32x2 w;
      w[0] = pack_bf16x2(o[rb][dt][0] * inv, o[rb][dt][1] * inv);
      w[1] = pack_bf16x2(o[rb][dt][2] * inv, o[rb][dt][3] * inv);
      *(u32x2 *)(wo + dt * 16) = w;
    }
    if (lane < 16) *(f32x2 *)(a.ws_ml + slot * 2) = f32x2{m_ref[rb], l_tot[rb]};
  }
}

// Merges the chunk partials of every split (request, kv-head, row tile):
// with w_c = l_c 2^((m_c - m) c), out = sum_c w_c o_c / sum_c w_c, o_c being
// chunk c's own normalised output.  One workgroup per 16 rows of one
// kv-head; each thread owns D/16 columns of one row.  With a plan table the
// grid holds the split requests' rows only (group_end counts 16-row merge
// blocks); without one, workgroup b takes rows (b % 8) * 16 .. +15 of
// (kv-head, row tile) group b / 8 in the scan order, and the workgroups of
// unsplit requests or past a tile's rows return at once.
template <int D>
__global__ __launch_bounds__(kThreads) void tree_attn_combine_kernel(TreeAttnArgs a) {
  constexpr int kRowsPerWg = 16;
  constexpr int TPR = kThreads / kRowsPerWg;  // threads per row
  constexpr int CPT = D / TPR;                // columns per thread (8 or 4)
  if ((int64_t)blockIdx.x >= a.merge_blocks) {
    // fused verification step: one acceptance wave per request after the
    // merge workgroups (the argmax finished in the previous launch)
    __shared__ int32_t acc_lds[kThreads / 64][3][kMaxTreeNodes];
    const int w = threadIdx.x >> 6;
    const int64_t r = ((int64_t)blockIdx.x - a.merge_blocks) * (kThreads / 64) + w;
    if (r < a.accept_requests)
      accept_request((int)r, a.total_nodes, a.node_indptr, a.parent, a.draft_tokens, a.argmax_out, a.max_accept,
                     a.accept_len, a.accept_tokens, a.accept_nodes, acc_lds[w][0], acc_lds[w][1], acc_lds[w][2]);
    return;
  }
  int32_t node_base, n, L, chunk_len, tile, g, rl;
  int64_t ubase;
  const int G = a.group, RT = a.rows_per_tile;
  if (a.plan_count > 0) {
    const int lo = __builtin_amdgcn_readfirstlane(find_plan_entry(a, blockIdx.x, true));
    if (lo < 0) return;
    const int64_t mbase = lo > 0 ? a.plan[lo - 1].group_end : 0;
    ubase = lo > 0 ? a.plan[lo - 1].unit_end : 0;
    node_base = a.plan[lo].node_base;
    n = plan_nodes(a.plan[lo].n_and_len);
    L = plan_prefix_len(a.plan[lo].n_and_len);
    chunk_len = plan_chunk_keys(a.plan[lo].request_and_chunk);
    const int32_t per_head = ceil_div(n * G, kRowsPerWg);
    if (per_head <= 0) return;
    const int32_t local = (int32_t)(blockIdx.x - mbase);
    g = local / per_head;
    const int32_t row = (local - g * per_head) * kRowsPerWg + (int)threadIdx.x / TPR;
    if (g >= a.num_kv_heads || row >= n * G) return;
    tile = row / RT;
    rl = row - tile * RT;
  } else {
    const int64_t gid = blockIdx.x / (kMaxRowsPerTile / kRowsPerWg);
    const int rblk = blockIdx.x % (kMaxRowsPerTile / kRowsPerWg);
    if (gid >= a.row_groups) return;
    int32_t r;
    int64_t gbase;
    if (!locate_request(gid, true, a, r, ubase, gbase)) return;
    node_base = a.node_indptr[r];
    n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
    L = max(a.prefix_len[r], 0);
    chunk_len = chunk_keys(n, G, RT, a.chunk_target, a.chunk_floor);
    if (n == 0) return;
    const int32_t tiles_r = row_tiles(n, G, RT);
    const int64_t u = gid - gbase;
    tile = (int32_t)(u % tiles_r);
    g = (int32_t)(u / tiles_r);
    rl = rblk * kRowsPerWg + (int)threadIdx.x / TPR;
    if (rl >= min(RT, n * G - tile * RT)) return;
  }
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  if (chunk_len <= 0 || chunk_len > kMaxChunk || chunk_len % kKeysPerBlock != 0) return;
  const int32_t tiles = row_tiles(n, G, RT);
  const int32_t chunks = prefix_chunks(L, chunk_len);
  if (chunks == 1) return;
  const int col = ((int)threadIdx.x % TPR) * CPT;
  const float c = a.scale_log2;
  float mm = -1e30f, ll = 0.f;
  f32x4 acc[CPT / 4];
#pragma unroll
  for (int k = 0; k < CPT / 4; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int cc = 0; cc < chunks; ++cc) {
    const int64_t slot = (ubase + ((int64_t)cc * a.num_kv_heads + g) * tiles + tile) * kMaxRowsPerTile + rl;
    const f32x2 ml = *(const f32x2 *)(a.ws_ml + slot * 2);
    u32x4 raw = {0u, 0u, 0u, 0u};  // CPT bf16 values
    if (CPT == 8) raw = *(const u32x4 *)(a.ws_o + slot * D + col);
    else { const u32x2 h = *(const u32x2 *)(a.ws_o + slot * D + col); raw[0] = h[0]; raw[1] = h[1]; }
    const float m_new = fmaxf(mm, ml[0]);
    const float sa = __builtin_amdgcn_exp2f((mm - m_new) * c);
    const float wb = ml[1] * __builtin_amdgcn_exp2f((ml[0] - m_new) * c);
    mm = m_new;
    ll = ll * sa + wb;
#pragma unroll
    for (int k = 0; k < CPT / 4; ++k) {
      const f32x4 v = {bf16_bits_to_float(raw[2 * k] & 0xffffu), bf16_bits_to_float(raw[2 * k] >> 16),
                       bf16_bits_to_float(raw[2 * k + 1] & 0xffffu), bf16_bits_to_float(raw[2 * k + 1] >> 16)};
      acc[k] = acc[k] * sa + v * wb;
    }
  }
  const float inv = ll > 0.f ? 1.f / ll : 0.f;
  const int row = tile * RT + rl;
  const int node = row / G, hh = row - (row / G) * G;
  __bf16 *op = (__bf16 *)a.out + ((int64_t)(node_base + node) * a.num_q_heads + g * G + hh) * D + col;
#pragma unroll
  for (int k = 0; k < CPT / 4; ++k) {
    u32x2 w;
    w[0] = pack_bf16x2(acc[k][0] * inv, acc[k][1] * inv);
    w[1] = pack_bf16x2(acc[k][2] * inv, acc[k][3] * inv);
    *(u32x2 *)(op + 4 * k) = w;
  }
}

// fp32 path: one workgroup per (node, q-head), exact fp32 arithmetic on the
// vector ALUs (small shapes; the matrix cores have no fp32 input path that
// keeps full precision for Q.K).  The node's keys -- its prefix, then its
// root path -- are taken in chunks of 1024: every thread scores whole keys
// (a dot product over the head dim), the chunk's softmax weights go to LDS,
// then thread (group g, column d) accumulates column d of the weighted
// values over every G-th key; an online softmax joins the chunks.
template <int D>
__global__ __launch_bounds__(256) void tree_attn_f32_kernel(TreeAttnArgs a) {
  constexpr int kT = 256;
  constexpr int G = kT / D;       // key groups of the value accumulation
  constexpr int CH = 1024;        // keys per chunk
  __shared__ float qs[D];
  __shared__ float ps[CH];
  __shared__ int64_t rowoff[CH];  // >= 0: element offset in the page pool; -1: zero key; <= -2: tree row
  __shared__ int32_t path[kMaxTreeNodes];
  __shared__ float red[kT / 64];
  __shared__ float part[kT];
  __shared__ int32_t info[4];     // request, node base, path length, ok
  const int64_t idx = blockIdx.x;
  const int32_t node = (int32_t)(idx / a.num_q_heads);
  const int32_t h = (int32_t)(idx % a.num_q_heads);
  if (node >= a.total_nodes) return;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if (t == 0) {
    // request owning this node, then the node's root path
    int lo = 0, hi = a.num_requests - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.node_indptr[mid] <= node) lo = mid; else hi = mid - 1;
    }
    const int32_t base = a.node_indptr[lo];
    const int32_t n = a.node_indptr[lo + 1] - base;
    int ok = node >= base && node < base + n && n <= kMaxTreeNodes;
    int len = 0;
    if (ok) {
      int v = node - base;
      for (int step = 0; step < kMaxTreeNodes; ++step) {
        path[len++] = v;
        if (v == 0) break;
        const int p = a.parent[base + v];
        if (p < 0 || p >= v) break;
        v = p;
      }
    }
    info[0] = lo;
    info[1] = base;
    info[2] = len;
    info[3] = ok;
  }
  const int g = h / a.group;
  const float *q = (const float *)a.q + ((int64_t)node * a.num_q_heads + h) * D;
  for (int d = t; d < D; d += kT) qs[d] = q[d];
  __syncthreads();
  if (!info[3]) return;
  const int r = info[0], base = info[1], npath = info[2];
  const int32_t L = max(a.prefix_len[r], 0);
  const int32_t nkeys = L + npath;
  const float *kp = (const float *)a.k_pages, *vp = (const float *)a.v_pages;
  const float *kt = (const float *)a.k_tree, *vt = (const float *)a.v_tree;
  const int col = t % D, grp = t / D;
  float m = -INFINITY, l = 0.f, acc = 0.f;
  for (int32_t k0 = 0; k0 < nkeys; k0 += CH) {
    const int n = min(CH, nkeys - k0);
    float cmax = -INFINITY;
    for (int j = t; j < n; j += kT) {
      const int32_t key = k0 + j;
      int64_t off;
      const float *kr;
      if (key < L) {
        const int32_t e = key / kPageSize;
        const int32_t pg = e < a.bt_stride ? a.block_table[(int64_t)r * a.bt_stride + e] : -1;
        off = (pg < 0 || pg >= a.num_pages) ? -1
              : (((int64_t)pg * a.num_kv_heads + g) * kPageSize + key % kPageSize) * D;
        kr = off >= 0 ? kp + off : nullptr;
      } else {
        const int64_t toff = ((int64_t)(base + path[key - L]) * a.num_kv_heads + g) * D;
        off = -2 - toff;
        kr = kt + toff;
      }
      float sc = 0.f;
      if (kr) {
#pragma unroll
        for (int d = 0; d < D; d += 4) {
          const f32x4 kv = *(const f32x4 *)(kr + d);
          sc = fmaf(qs[d], kv[0], sc);
          sc = fmaf(qs[d + 1], kv[1], sc);
          sc = fmaf(qs[d + 2], kv[2], sc);
          sc = fmaf(qs[d + 3], kv[3], sc);
        }
      }
      sc *= a.sm_scale;
      ps[j] = sc;
      rowoff[j] = off;
      cmax = fmaxf(cmax, sc);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cmax = fmaxf(cmax, __shfl_xor(cmax, o, 64));
    if (lane == 0) red[wave] = cmax;
    __syncthreads();
    float mn = m;
#pragma unroll
    for (int w = 0; w < kT / 64; ++w) mn = fmaxf(mn, red[w]);
    __syncthreads();
    const float alpha = m > -INFINITY ? expf(m - mn) : 0.f;
    float lsum = 0.f;
    for (int j = t; j < n; j += kT) {
      const float p = expf(ps[j] - mn);
      ps[j] = p;
      lsum += p;
    }
    lsum = wave_sum(lsum);
    if (lane == 0) red[wave] = lsum;
    __syncthreads();
    float csum = 0.f;
#pragma unroll
    for (int w = 0; w < kT / 64; ++w) csum += red[w];
    l = l * alpha + csum;
    acc *= alpha;
    m = mn;
    if (grp < G)
      for (int j0 = grp; j0 < n; j0 += 8 * G) {
        // eight keys' loads in flight before their products
        float pv[8], vv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u * G;
          const int64_t off = j < n ? rowoff[j] : -1;
          const float *src = off >= 0 ? vp + off + col : off == -1 ? vt + col : vt + (-2 - off) + col;
          pv[u] = j < n && off != -1 ? ps[j] : 0.f;
          vv[u] = *src;  // a zero row reads tree row 0 and weighs it 0 below
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = pv[u] != 0.f ? fmaf(pv[u], vv[u], acc) : acc;
      }
    __syncthreads();  // ps, rowoff and red are rewritten by the next chunk
  }
  part[t] = acc;
  __syncthreads();
  if (t < D) {
    float o = 0.f;
#pragma unroll
    for (int k = 0; k < G; ++k) o += part[k * D + t];
    float *out = (float *)a.out + ((int64_t)node * a.num_q_heads + h) * D;
    out[t] = l > 0.f ? o / l : 0.f;
  }
}

}  // namespace

// Split-KV partial results of adaserve_tree_attn_verify_noalloc, for callers
// that cannot allocate: every call on a device shares that device's copy.
// The kernels take its device address (from hipGetSymbolAddress, below) as
// their workspace pointer, exactly like a caller's workspace; the array's
// name is only a host-side stand-in and is never passed to a kernel.
static __device__ __align__(256) unsigned char scratch[ADASERVE_TREE_ATTN_SCRATCH_BYTES];

hipError_t tree_attn_scratch(void **out) {
  static std::mutex mu;
  static void *addr[256];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 256) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (uintptr_t)p % 256 != 0) return hipErrorInvalidValue;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

// Device address of g_zero16 on the current device, looked up once per device.
static hipError_t zero16_address(const void **out) {
  static std::mutex mu;
  static const void *addr[256];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 256) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_zero16));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

// The attention grid (and, in the one-call step, the argmax workgroups after
// it) with the K/V load hint the plan chose.
static void launch_attention(const TreeAttnArgs &a, int head_dim, int64_t blocks, hipStream_t stream) {
  const dim3 grid((unsigned)blocks), block(kThreads);
  if (head_dim == 128) {
    if (a.stream_kv)
      hipLaunchKernelGGL((tree_attn_bf16_kernel<128, true>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((tree_attn_bf16_kernel<128, false>), grid, block, 0, stream, a);
  } else {
    if (a.stream_kv)
      hipLaunchKernelGGL((tree_attn_bf16_kernel<64, true>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((tree_attn_bf16_kernel<64, false>), grid, block, 0, stream, a);
  }
}

hipError_t launch_tree_attn_bf16(TreeAttnArgs &a, int head_dim, bool needs_combine, hipStream_t stream) {
  if (a.units == 0) return hipSuccess;
  hipError_t e = zero16_address(&a.zero16);
  if (e != hipSuccess) return e;
  const dim3 block(kThreads);
  launch_attention(a, head_dim, a.padded_grid, stream);
  e = hipGetLastError();
  if (e != hipSuccess || !needs_combine) return e;
  const dim3 cgrid((unsigned)a.merge_blocks);
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_combine_kernel<128>, cgrid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_combine_kernel<64>, cgrid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_verify_step_bf16(TreeAttnArgs &a, int head_dim, bool needs_combine, hipStream_t stream) {
  hipError_t e = zero16_address(&a.zero16);
  if (e != hipSuccess) return e;
  const dim3 block(kThreads);
  const int64_t g1 = (a.units > 0 ? a.padded_grid : 0) + a.argmax_rows;
  if (a.units == 0) a.padded_grid = 0;
  if (g1 > 0) {
    launch_attention(a, head_dim, g1, stream);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (!needs_combine) a.merge_blocks = 0;
  const int64_t g2 = a.merge_blocks + (a.accept_requests + kThreads / 64 - 1) / (kThreads / 64);
  if (g2 == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_combine_kernel<128>, dim3((unsigned)g2), block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_combine_kernel<64>, dim3((unsigned)g2), block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_tree_attn_f32(const TreeAttnArgs &a, int head_dim, hipStream_t stream) {
  const int64_t blocks = (int64_t)a.total_nodes * a.num_q_heads;
  if (blocks == 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(256);
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_f32_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_f32_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
