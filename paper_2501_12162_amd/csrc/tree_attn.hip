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
//    global_load_lds (no staging registers) into a 4-stage ring: three
//    blocks are in flight while one is multiplied, one barrier per block,
//    waits counted by hand (vmcnt) so the ring really overlaps;
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
//    its partial (reference max, denominator, numerator) and a second,
//    fully parallel kernel merges them (the kernel boundary makes the
//    partials of every XCD visible without per-workgroup cache flushes).
#include <mutex>

#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace adaserve {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxChunkPages = kMaxChunk / kPageSize;

// 16 bytes of zeros: the source of every DMA lane whose key is out of range,
// so no NaN from an unused page slot reaches LDS.  Its device address is
// passed in the kernel arguments (resolved once per device on the host).
__device__ __align__(16) uint32_t g_zero16[4];

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void global_void_t;

// 16 bytes from `src` (per lane) to LDS at `wave_dst` + 16 * lane.
__device__ __forceinline__ void dma16(const void *src, void *wave_dst) {
  __builtin_amdgcn_global_load_lds((global_void_t *)src, (lds_void_t *)wave_dst, 16, 0, 0);
}

// s_waitcnt encodings (gfx9): vmcnt(N) with the other counters left open,
// and lgkmcnt(0) with vmcnt left open.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0xF70 | N);
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

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

template <int D>
__global__ __launch_bounds__(kThreads, 2) void tree_attn_bf16_kernel(TreeAttnArgs a) {
  constexpr int KS = D / 32;                 // MFMA k-steps over the head dim
  constexpr int DT = D / 16;                 // 16-wide output tiles over the head dim
  constexpr int KB = kKeysPerBlock;          // 32 keys per pipeline stage
  constexpr int NSTAGE = 4;
  constexpr int ROWB = D * 2;                // bytes per key row
  constexpr int NCH = D / 8;                 // 16-byte chunks per key row
  constexpr int BLK = KB * ROWB;             // bytes of K (or V) per stage
  constexpr int WI = BLK / 1024 / 4;         // DMA wave-instructions per wave per tensor
  constexpr int RPI = 1024 / ROWB;           // key rows covered by one wave-instruction
  constexpr int NDMA = 2 * WI;               // DMA instructions per thread per block
  constexpr float kRescaleLog2 = 8.f;

  // Four pipeline stages, each [K|V][32 keys][D], as separate LDS objects so
  // the compiler can tell a stage being filled from the stage being read and
  // does not wait for every in-flight load before each read.
  __shared__ __align__(1024) char st0[2 * BLK];
  __shared__ __align__(1024) char st1[2 * BLK];
  __shared__ __align__(1024) char st2[2 * BLK];
  __shared__ __align__(1024) char st3[2 * BLK];
  __shared__ __align__(16) uint32_t anc[kMaxTreeNodes * 4];
  __shared__ int32_t pages[kMaxChunkPages];
  __shared__ int32_t par[kMaxTreeNodes];

  const int64_t uid = xcd_swizzle(blockIdx.x, a.padded_grid);
  if (uid >= a.units) return;
  int32_t r, node_base, n, L;
  int64_t ubase;
  if (a.plan_count > 0) {
    // binary search of the dispatch-ordered plan in the kernel arguments
    int lo = 0, hi = a.plan_count - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (a.plan[mid].unit_end > uid) hi = mid; else lo = mid + 1;
    }
    if (a.plan[lo].unit_end <= uid) return;
    r = a.plan[lo].request;
    ubase = lo > 0 ? a.plan[lo - 1].unit_end : 0;
    node_base = a.plan[lo].node_base;
    n = a.plan[lo].n_and_len & 0xff;
    L = a.plan[lo].n_and_len >> 8;
  } else {
    int64_t gbase;
    if (!locate_request(uid, false, a, r, ubase, gbase)) return;
    node_base = a.node_indptr[r];
    n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
    L = max(a.prefix_len[r], 0);
  }
  // Request values are uniform; make that visible so branches on them stay scalar.
  r = __builtin_amdgcn_readfirstlane(r);
  node_base = __builtin_amdgcn_readfirstlane(node_base);
  n = __builtin_amdgcn_readfirstlane(n);
  L = __builtin_amdgcn_readfirstlane(L);
  ubase = ((int64_t)__builtin_amdgcn_readfirstlane((int32_t)(ubase >> 32)) << 32) |
          (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)ubase);
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.group;
  const int RT = a.rows_per_tile;
  const int32_t tiles = row_tiles(n, G, RT);
  const int32_t chunk_len = chunk_keys(n, G, RT, a.chunk_target, a.chunk_floor);
  const int32_t chunks = prefix_chunks(L, chunk_len);
  const int64_t u = uid - ubase;
  const int32_t tile = (int32_t)(u % tiles);
  const int64_t rest = u / tiles;
  const int32_t chunk = (int32_t)(rest % chunks);
  const int32_t g = (int32_t)(rest / chunks);
  const int32_t M = n * G;
  const int32_t row0 = tile * RT;
  const int32_t row_end = min(M, row0 + RT);
  const bool last_chunk = chunk == chunks - 1;
  const int32_t k0 = chunk * chunk_len;
  const int32_t k1 = min(L, k0 + chunk_len);
  const int32_t n_prefix_blocks = k1 > k0 ? ceil_div(k1 - k0, KB) : 0;
  const int32_t n_tree_blocks = last_chunk ? ceil_div(n, KB) : 0;
  const int32_t n_blocks = n_prefix_blocks + n_tree_blocks;
  const int32_t page0 = k0 / kPageSize;
  const int32_t npages = k1 > k0 ? ceil_div(k1, kPageSize) - page0 : 0;

  // ---- start-up: block table, parents and queries, all loads in flight together
  for (int i = tid; i < npages; i += kThreads) {
    int32_t p = -1;
    if (page0 + i < a.bt_stride) {
      p = a.block_table[(int64_t)r * a.bt_stride + page0 + i];
      if (p < 0 || p >= a.num_pages) p = -1;
    }
    pages[i] = p;
  }
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

  // ---- DMA addressing: wave-instruction i of this wave fills LDS bytes
  // [(wave*WI + i)*1024, +1024) of a K (or V) stage; lane `lane` lands on key
  // row dma_row[i], slot `slot`, so it fetches chunk slot ^ swizzle(row).
  // A wave's rows lie in one 16-key page (wave_page of the two in a block),
  // so the page and its base address are wave-uniform; lanes add a 32-bit
  // byte offset inside the (page, kv-head) chunk or inside the tree block.
  const int slot = ((lane * 16) % ROWB) / 16;
  const int wave_page = (wave * WI * RPI) / kPageSize;
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
  const char *kpg = (const char *)a.k_pages + (int64_t)g * kPageSize * D * 2;
  const char *vpg = (const char *)a.v_pages + (int64_t)g * kPageSize * D * 2;
  const char *ktr = (const char *)a.k_tree + ((int64_t)node_base * a.num_kv_heads + g) * D * 2;
  const char *vtr = (const char *)a.v_tree + ((int64_t)node_base * a.num_kv_heads + g) * D * 2;
  auto issue = [&](char *stage_dst, int blk) {
    char *kdst = stage_dst;
    char *vdst = kdst + BLK;
    const char *kb, *vb;
    int rows_left;
    const bool pre = blk < n_prefix_blocks;
    if (pre) {
      const int32_t p = __builtin_amdgcn_readfirstlane(pages[blk * (KB / kPageSize) + wave_page]);
      rows_left = p >= 0 ? k1 - k0 - blk * KB : 0;
      kb = kpg + (int64_t)max(p, 0) * page_stride_b;
      vb = vpg + (int64_t)max(p, 0) * page_stride_b;
    } else {
      const int tb = blk - n_prefix_blocks;
      rows_left = n - tb * KB;
      kb = ktr + (int64_t)tb * KB * tree_stride * 2;
      vb = vtr + (int64_t)tb * KB * tree_stride * 2;
    }
    if (rows_left >= KB) {
#pragma unroll
      for (int i = 0; i < WI; ++i) {
        const uint32_t off = pre ? page_off[i] : tree_off[i];
        dma16(kb + off, kdst + (wave * WI + i) * 1024);
        dma16(vb + off, vdst + (wave * WI + i) * 1024);
      }
    } else {
#pragma unroll
      for (int i = 0; i < WI; ++i) {
        const uint32_t off = pre ? page_off[i] : tree_off[i];
        const bool ok = dma_row[i] < rows_left;
        dma16(ok ? (const void *)(kb + off) : a.zero16, kdst + (wave * WI + i) * 1024);
        dma16(ok ? (const void *)(vb + off) : a.zero16, vdst + (wave * WI + i) * 1024);
      }
    }
  };


  __syncthreads();  // pages[] and par[] visible
  if (n_blocks > 0) issue(st0, 0);
  if (n_blocks > 1) issue(st1, 1);
  if (n_blocks > 2) issue(st2, 2);

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
  int koff[KS];  // K fragment for keys kt*16 + j16 (add kt*16*ROWB), chunk ks*4 + q
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = j16 * ROWB + (((ks * 4 + q) ^ swizzle<NCH>(j16)) * 16);
  int voff[DT];  // transposed V read: key row q*4 + (j16 >> 2) (+16 for the upper half)
  {
    const int vrow = q * 4 + (j16 >> 2);
    const int sw = swizzle<NCH>(vrow);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      voff[dt] = BLK + vrow * ROWB + (((dt * 2 + ((j16 & 3) >> 1)) ^ sw) * 16) + (j16 & 1) * 8;
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

  // One pipeline step: wait for block blk (at most min(2, n_blocks-1-blk)
  // younger blocks of this wave may still be in flight), barrier (the block
  // is complete in LDS and every wave has finished reading the stage that
  // block blk+3 will fill), issue block blk+3, multiply block blk.
  auto compute = [&](const char *stage, int blk) {
    const bool tree_blk = blk >= n_prefix_blocks;
    const int tb = blk - n_prefix_blocks;
    const int valid = tree_blk ? min(KB, n - tb * KB) : min(KB, k1 - k0 - blk * KB);
    const bool need_mask = tree_blk || valid < KB;

    // S^T tiles: s[rb][kt] holds keys kt*16 + q*4 + e of row j16.
    f32x4 s[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[0][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[1][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = *(const bf16x8 *)(stage + koff[ks] + kt * 16 * ROWB);
        s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[0][ks], s[0][kt], 0, 0, 0);
        s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[1][ks], s[1][kt], 0, 0, 0);
      }
    }

    bf16x8 pk[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      if (need_mask) {
        uint32_t aw = 0xffffffffu;
        if (tree_blk) {
          const int node = min((wrow0 + rb * 16 + j16) / G, n - 1);
          aw = anc[node * 4 + tb];
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
      float bm = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(s[rb][0][0], s[rb][0][1]), s[rb][0][2]),
                                 __builtin_fmaxf(s[rb][0][3], s[rb][1][0]));
      bm = __builtin_fmaxf(__builtin_fmaxf(bm, s[rb][1][1]), __builtin_fmaxf(s[rb][1][2], s[rb][1][3]));
      bm = max_over_lane_rows(bm);
      const bool up = bm > m_ref[rb] + up_raw;
      if (__any(up)) {
        const float m_new = up ? bm : m_ref[rb];
        const float alpha = up ? __builtin_amdgcn_exp2f((m_ref[rb] - m_new) * c) : 1.f;
        m_ref[rb] = m_new;
        osum[rb] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[rb][dt] *= alpha;
      }
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

    // O^T += V^T P^T.  k-slot (q, e) of the A operand is key q*4 + e (e < 4)
    // or 16 + q*4 + (e - 4): the keys the packed P fragment carries.  The
    // transposed read hands lane (q, j16) V[kbase + e][dt*16 + j16], e < 4.
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(stage + voff[dt]));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(stage + voff[dt] + 16 * ROWB));
      const bf16x8 vf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[0], o[0][dt], 0, 0, 0);
      o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[1], o[1][dt], 0, 0, 0);
    }
    osum[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pk[0], osum[0], 0, 0, 0);
    osum[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pk[1], osum[1], 0, 0, 0);
  };
  auto step = [&](const char *cur, char *refill, int blk) {
    const int younger = min(NSTAGE - 2, n_blocks - 1 - blk);
    if (younger >= 2) wait_vmcnt<2 * NDMA>();
    else if (younger == 1) wait_vmcnt<NDMA>();
    else wait_vmcnt<0>();
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    if (blk + NSTAGE - 1 < n_blocks) issue(refill, blk + NSTAGE - 1);
    if (wave_live) compute(cur, blk);
  };
  for (int blk = 0; blk < n_blocks; blk += NSTAGE) {
    step(st0, st3, blk);
    if (blk + 1 >= n_blocks) break;
    step(st1, st0, blk + 1);
    if (blk + 2 >= n_blocks) break;
    step(st2, st1, blk + 2);
    if (blk + 3 >= n_blocks) break;
    step(st3, st2, blk + 3);
  }

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

  // ---- split prefix: write this chunk's partial (reference max, denominator,
  // numerator); tree_attn_combine_kernel merges the chunks after this kernel.
  if (!wave_live) return;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = wrow0 + rb * 16 + j16;
    if (row >= row_end) continue;
    const int64_t slot = uid * kMaxRowsPerTile + (row - row0);
    float *wo = a.ws_o + slot * D + q4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(f32x4 *)(wo + dt * 16) = o[rb][dt];
    if (lane < 16) *(f32x2 *)(a.ws_ml + slot * 2) = f32x2{m_ref[rb], l_tot[rb]};
  }
}

// Finds the request of (kv-head, row tile) group `gid` from the plan in the
// kernel arguments, or by scanning the device arrays.
__device__ __forceinline__ bool group_request(const TreeAttnArgs &a, int64_t gid, int32_t &node_base,
                                              int32_t &n, int32_t &L, int64_t &ubase, int64_t &gbase) {
  if (a.plan_count > 0) {
    int lo = 0, hi = a.plan_count - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (a.plan[mid].group_end > gid) hi = mid; else lo = mid + 1;
    }
    if (a.plan[lo].group_end <= gid) return false;
    ubase = lo > 0 ? a.plan[lo - 1].unit_end : 0;
    gbase = lo > 0 ? a.plan[lo - 1].group_end : 0;
    node_base = a.plan[lo].node_base;
    n = a.plan[lo].n_and_len & 0xff;
    L = a.plan[lo].n_and_len >> 8;
    return true;
  }
  int32_t r;
  if (!locate_request(gid, true, a, r, ubase, gbase)) return false;
  node_base = a.node_indptr[r];
  n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
  L = max(a.prefix_len[r], 0);
  return true;
}

// Merges the chunk partials of every split (request, kv-head, row tile):
// out = sum_c 2^((m_c - m) c) o_c / sum_c 2^((m_c - m) c) l_c.  One workgroup
// per 16 rows of a group; each thread owns 8 columns of one row.
template <int D>
__global__ __launch_bounds__(kThreads) void tree_attn_combine_kernel(TreeAttnArgs a) {
  constexpr int kRowsPerWg = 16;
  constexpr int TPR = kThreads / kRowsPerWg;  // threads per row
  constexpr int CPT = D / TPR;                // columns per thread (8 or 4)
  const int64_t gid = blockIdx.x / (kMaxRowsPerTile / kRowsPerWg);
  const int rblk = blockIdx.x % (kMaxRowsPerTile / kRowsPerWg);
  if (gid >= a.row_groups) return;
  int32_t node_base, n, L;
  int64_t ubase, gbase;
  if (!group_request(a, gid, node_base, n, L, ubase, gbase)) return;
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  const int G = a.group, RT = a.rows_per_tile;
  const int32_t tiles = row_tiles(n, G, RT);
  const int32_t chunks = prefix_chunks(L, chunk_keys(n, G, RT, a.chunk_target, a.chunk_floor));
  if (chunks == 1) return;
  const int64_t u = gid - gbase;
  const int32_t tile = (int32_t)(u % tiles);
  const int32_t g = (int32_t)(u / tiles);
  const int rl = rblk * kRowsPerWg + (int)threadIdx.x / TPR;
  const int rows = min(RT, n * G - tile * RT);
  if (rl >= rows) return;
  const int col = ((int)threadIdx.x % TPR) * CPT;
  const float c = a.scale_log2;
  float mm = -1e30f, ll = 0.f;
  f32x4 acc[CPT / 4];
#pragma unroll
  for (int k = 0; k < CPT / 4; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int cc = 0; cc < chunks; ++cc) {
    const int64_t slot = (ubase + ((int64_t)g * chunks + cc) * tiles + tile) * kMaxRowsPerTile + rl;
    const f32x2 ml = *(const f32x2 *)(a.ws_ml + slot * 2);
    const float m_new = fmaxf(mm, ml[0]);
    const float sa = __builtin_amdgcn_exp2f((mm - m_new) * c);
    const float sb = __builtin_amdgcn_exp2f((ml[0] - m_new) * c);
    mm = m_new;
    ll = ll * sa + ml[1] * sb;
#pragma unroll
    for (int k = 0; k < CPT / 4; ++k)
      acc[k] = acc[k] * sa + *(const f32x4 *)(a.ws_o + slot * D + col + 4 * k) * sb;
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

// fp32 path: one wave per (node, q-head), exact fp32 arithmetic on the
// vector ALUs (small shapes; the matrix cores have no fp32 input path that
// keeps full precision for Q.K).
template <int D>
__global__ __launch_bounds__(64) void tree_attn_f32_kernel(TreeAttnArgs a) {
  constexpr int PER = D / 64;
  const int64_t idx = blockIdx.x;
  const int32_t node = (int32_t)(idx / a.num_q_heads);
  const int32_t h = (int32_t)(idx % a.num_q_heads);
  if (node >= a.total_nodes) return;
  const int lane = threadIdx.x;
  // request owning this node
  int lo = 0, hi = a.num_requests - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.node_indptr[mid] <= node) lo = mid; else hi = mid - 1;
  }
  const int r = lo;
  const int32_t base = a.node_indptr[r];
  const int32_t n = a.node_indptr[r + 1] - base;
  if (node < base || node >= base + n || n > kMaxTreeNodes) return;
  const int32_t L = max(a.prefix_len[r], 0);
  const int g = h / a.group;
  const float *q = (const float *)a.q + ((int64_t)node * a.num_q_heads + h) * D;
  float qv[PER], acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    qv[i] = q[lane + 64 * i];
    acc[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  auto visit = [&](const float *kp, const float *vp) {
    float s = 0.f;
    if (kp) {
#pragma unroll
      for (int i = 0; i < PER; ++i) s += qv[i] * kp[lane + 64 * i];
    }
    s = wave_sum(s) * a.sm_scale;
    const float m_new = fmaxf(m, s);
    const float alpha = expf(m - m_new);
    const float p = expf(s - m_new);
    l = l * alpha + p;
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = acc[i] * alpha + (vp ? p * vp[lane + 64 * i] : 0.f);
    m = m_new;
  };
  for (int32_t t = 0; t < L; ++t) {
    int32_t p = t / kPageSize < a.bt_stride ? a.block_table[(int64_t)r * a.bt_stride + t / kPageSize] : -1;
    if (p < 0 || p >= a.num_pages) {
      visit(nullptr, nullptr);
    } else {
      const int64_t off = (((int64_t)p * a.num_kv_heads + g) * kPageSize + t % kPageSize) * D;
      visit((const float *)a.k_pages + off, (const float *)a.v_pages + off);
    }
  }
  int v = node - base;
  for (int step = 0; step < kMaxTreeNodes; ++step) {
    const int64_t off = ((int64_t)(base + v) * a.num_kv_heads + g) * D;
    visit((const float *)a.k_tree + off, (const float *)a.v_tree + off);
    if (v == 0) break;
    const int p = a.parent[base + v];
    if (p < 0 || p >= v) break;
    v = p;
  }
  float *o = (float *)a.out + ((int64_t)node * a.num_q_heads + h) * D;
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) o[lane + 64 * i] = acc[i] * inv;
}

}  // namespace

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

hipError_t launch_tree_attn_bf16(TreeAttnArgs &a, int head_dim, bool needs_combine, hipStream_t stream) {
  if (a.units == 0) return hipSuccess;
  hipError_t e = zero16_address(&a.zero16);
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)a.padded_grid), block(kThreads);
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_bf16_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_bf16_kernel<64>, grid, block, 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess || !needs_combine) return e;
  const dim3 cgrid((unsigned)(a.row_groups * (kMaxRowsPerTile / 16)));
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_combine_kernel<128>, cgrid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_combine_kernel<64>, cgrid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_tree_attn_f32(const TreeAttnArgs &a, int head_dim, hipStream_t stream) {
  const int64_t blocks = (int64_t)a.total_nodes * a.num_q_heads;
  if (blocks == 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(64);
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_f32_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_f32_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
