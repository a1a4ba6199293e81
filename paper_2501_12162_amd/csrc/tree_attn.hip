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
//  * K/V are staged in LDS 64 keys at a time: the next block is loaded into
//    registers while the current block is multiplied;
//  * S^T = K Q^T and O^T = V^T P^T run on v_mfma_f32_16x16x32_bf16.  In this
//    orientation a lane owns one query row, so the online softmax needs no
//    cross-lane traffic except a max over the four 16-lane rows, and V is
//    read transposed straight from its natural layout with ds_read_b64_tr_b16;
//  * the tree block (the request's own N_r nodes) is one more K/V block
//    masked by 128-bit ancestor sets built in LDS from parent[];
//  * prefixes longer than one chunk are split across workgroups and the
//    partial (max, sum, numerator) triples are merged by a second kernel.
#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace adaserve {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxChunkPages = 512;  // chunk_keys <= 8192

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
      ng = (int64_t)a.num_kv_heads * row_tiles(n, a.group);
      nu = ng * prefix_chunks(L, a.chunk_keys);
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

template <int D>
__global__ __launch_bounds__(kThreads, 2) void tree_attn_bf16_kernel(TreeAttnArgs a) {
  constexpr int KS = D / 32;                            // MFMA k-steps over the head dim
  constexpr int DT = D / 16;                            // 16-wide output tiles over the head dim
  constexpr int KSTR = D + 8;                           // LDS row stride of K (elements)
  constexpr int VSTR = D + 16;                          // LDS row stride of V (elements)
  constexpr int TPK = D / 8;                            // threads per key row (16 B each)
  constexpr int KEYS_PER_LOAD = kThreads / TPK;
  constexpr int NLOAD = kKeysPerBlock / KEYS_PER_LOAD;

  __shared__ __align__(16) __bf16 k_lds[kKeysPerBlock * KSTR];
  __shared__ __align__(16) __bf16 v_lds[kKeysPerBlock * VSTR];
  __shared__ __align__(16) uint32_t anc[kMaxTreeNodes * 4];
  __shared__ int32_t pages[kMaxChunkPages];

  const int64_t uid = xcd_swizzle(blockIdx.x, a.padded_grid);
  if (uid >= a.units) return;
  int32_t r;
  int64_t ubase, gbase;
  if (!locate_request(uid, false, a, r, ubase, gbase)) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t node_base = a.node_indptr[r];
  const int32_t n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  const int32_t L = max(a.prefix_len[r], 0);
  const int G = a.group;
  const int32_t tiles = row_tiles(n, G);
  const int32_t chunks = prefix_chunks(L, a.chunk_keys);
  const int64_t u = uid - ubase;
  const int32_t tile = (int32_t)(u % tiles);
  const int64_t rest = u / tiles;
  const int32_t chunk = (int32_t)(rest % chunks);
  const int32_t g = (int32_t)(rest / chunks);
  const int32_t M = n * G;
  const int32_t row0 = tile * kRowsPerTile;
  const bool last_chunk = chunk == chunks - 1;
  const int32_t k0 = chunk * a.chunk_keys;
  const int32_t k1 = min(L, k0 + a.chunk_keys);
  const int32_t n_prefix_blocks = k1 > k0 ? ceil_div(k1 - k0, kKeysPerBlock) : 0;
  const int32_t n_tree_blocks = last_chunk ? ceil_div(n, kKeysPerBlock) : 0;
  const int32_t n_blocks = n_prefix_blocks + n_tree_blocks;
  const int32_t page0 = k0 / kPageSize;
  const int32_t npages = k1 > k0 ? ceil_div(k1, kPageSize) - page0 : 0;

  // Physical pages of this chunk (invalid ids become -1: read as zeros).
  for (int i = tid; i < npages; i += kThreads) {
    int32_t p = -1;
    if (page0 + i < a.bt_stride) {
      p = a.block_table[(int64_t)r * a.bt_stride + page0 + i];
      if (p < 0 || p >= a.num_pages) p = -1;
    }
    pages[i] = p;
  }
  // Ancestor sets: bit j of node i's set is 1 when j is on i's root-to-node
  // path (i included).  The walk stops at anything that is not a parent
  // strictly before its child, so malformed trees stay in bounds.
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
          const int p = a.parent[node_base + v];
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

  // Query fragments (B operand of S^T = K Q^T): lane holds row (lane & 15)
  // of each 16-row block, head-dim elements ks*32 + (lane >> 4)*8 .. +7.
  const int wrow0 = row0 + wave * 32;
  const bool wave_live = wrow0 < M;
  bf16x8 qf[2][KS];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = wrow0 + rb * 16 + (lane & 15);
    const bool valid = row < M;
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

  f32x4 o[2][DT];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[rb][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-1e30f, -1e30f};  // running max of this lane's row (log2 units)
  float l_run[2] = {0.f, 0.f};        // running denominator over this lane's keys

  u32x4 stk[NLOAD], stv[NLOAD];
  const int srow = tid / TPK;
  const int scol = (tid % TPK) * 8;
  auto stage = [&](int blk) {
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int kk = i * KEYS_PER_LOAD + srow;
      u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
      if (blk < n_prefix_blocks) {
        const int32_t t = k0 + blk * kKeysPerBlock + kk;
        if (t < k1) {
          const int32_t p = pages[t / kPageSize - page0];
          if (p >= 0) {
            const int64_t off = (((int64_t)p * a.num_kv_heads + g) * kPageSize + (t % kPageSize)) * D + scol;
            kv = *(const u32x4 *)((const __bf16 *)a.k_pages + off);
            vv = *(const u32x4 *)((const __bf16 *)a.v_pages + off);
          }
        }
      } else {
        const int j = (blk - n_prefix_blocks) * kKeysPerBlock + kk;
        if (j < n) {
          const int64_t off = ((int64_t)(node_base + j) * a.num_kv_heads + g) * D + scol;
          kv = *(const u32x4 *)((const __bf16 *)a.k_tree + off);
          vv = *(const u32x4 *)((const __bf16 *)a.v_tree + off);
        }
      }
      stk[i] = kv;
      stv[i] = vv;
    }
  };

  __syncthreads();  // pages[] and anc[] visible to every wave
  if (n_blocks > 0) stage(0);

  for (int blk = 0; blk < n_blocks; ++blk) {
    __syncthreads();  // every wave is done reading the previous block
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
      const int kk = i * KEYS_PER_LOAD + srow;
      *(u32x4 *)&k_lds[kk * KSTR + scol] = stk[i];
      *(u32x4 *)&v_lds[kk * VSTR + scol] = stv[i];
    }
    __syncthreads();
    if (blk + 1 < n_blocks) stage(blk + 1);
    if (!wave_live) continue;

    const bool tree_blk = blk >= n_prefix_blocks;
    const int tb = blk - n_prefix_blocks;
    const int valid = tree_blk ? min(kKeysPerBlock, n - tb * kKeysPerBlock)
                               : min(kKeysPerBlock, k1 - k0 - blk * kKeysPerBlock);

    // S^T tiles: s[rb][kt] holds keys kt*16 + (lane>>4)*4 + e of row (lane & 15).
    f32x4 s[2][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      s[0][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[1][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = *(const bf16x8 *)&k_lds[(kt * 16 + (lane & 15)) * KSTR + ks * 32 + (lane >> 4) * 8];
        s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[0][ks], s[0][kt], 0, 0, 0);
        s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[1][ks], s[1][kt], 0, 0, 0);
      }
    }

    bf16x8 pk[2][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      uint32_t aw0 = 0xffffffffu, aw1 = 0xffffffffu;
      if (tree_blk) {
        const int row = wrow0 + rb * 16 + (lane & 15);
        const int node = min(row / G, n - 1);
        aw0 = anc[node * 4 + tb * 2 + 0];
        aw1 = anc[node * 4 + tb * 2 + 1];
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = kt * 16 + (lane >> 4) * 4 + e;
          const int bit = (kt & 1) * 16 + (lane >> 4) * 4 + e;
          const uint32_t w = (kt < 2) ? aw0 : aw1;
          const bool ok = key < valid && ((w >> bit) & 1u);
          const float x = ok ? s[rb][kt][e] * a.scale_log2 : -INFINITY;
          s[rb][kt][e] = x;
          mx = fmaxf(mx, x);
        }
      }
      mx = max_over_lane_rows(mx);
      const float m_new = fmaxf(m_run[rb], mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run[rb] - m_new);
      m_run[rb] = m_new;
      float psum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = __builtin_amdgcn_exp2f(s[rb][kt][e] - m_new);
          s[rb][kt][e] = p;
          psum += p;
        }
      l_run[rb] = l_run[rb] * alpha + psum;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[rb][dt] *= alpha;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        u32x4 w;
        w[0] = pack_bf16x2(s[rb][2 * k2][0], s[rb][2 * k2][1]);
        w[1] = pack_bf16x2(s[rb][2 * k2][2], s[rb][2 * k2][3]);
        w[2] = pack_bf16x2(s[rb][2 * k2 + 1][0], s[rb][2 * k2 + 1][1]);
        w[3] = pack_bf16x2(s[rb][2 * k2 + 1][2], s[rb][2 * k2 + 1][3]);
        pk[rb][k2] = __builtin_bit_cast(bf16x8, w);
      }
    }

    // O^T += V^T P^T.  k-slot (q, e) of the A operand is key
    // k2*32 + q*4 + e (e < 4) or k2*32 + 16 + q*4 + (e - 4): the same keys
    // the packed P fragment carries.  The transposed LDS read hands lane
    // (q, j) the values V[kbase + e][dt*16 + j] for e = 0..3.
    {
      const int j = lane & 15, q = lane >> 4;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const int off0 = (k2 * 32 + q * 4 + (j >> 2)) * VSTR + dt * 16 + 4 * (j & 3);
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(v_lds + off0));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(v_lds + off0 + 16 * VSTR));
          u32x4 w;
          w[0] = __builtin_bit_cast(u32x2, lo)[0];
          w[1] = __builtin_bit_cast(u32x2, lo)[1];
          w[2] = __builtin_bit_cast(u32x2, hi)[0];
          w[3] = __builtin_bit_cast(u32x2, hi)[1];
          const bf16x8 vf = __builtin_bit_cast(bf16x8, w);
          o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[0][k2], o[0][dt], 0, 0, 0);
          o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pk[1][k2], o[1][dt], 0, 0, 0);
        }
      }
    }
  }

  if (!wave_live) return;
  const int q4 = (lane >> 4) * 4;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float l_tot = sum_over_lane_rows(l_run[rb]);
    const int row = wrow0 + rb * 16 + (lane & 15);
    if (row >= M) continue;
    if (chunks == 1) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      const int node = row / G, hh = row - (row / G) * G;
      __bf16 *op = (__bf16 *)a.out + ((int64_t)(node_base + node) * a.num_q_heads + g * G + hh) * D + q4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        u32x2 w;
        w[0] = pack_bf16x2(o[rb][dt][0] * inv, o[rb][dt][1] * inv);
        w[1] = pack_bf16x2(o[rb][dt][2] * inv, o[rb][dt][3] * inv);
        *(u32x2 *)(op + dt * 16) = w;
      }
    } else {
      const int64_t slot = uid * kRowsPerTile + (row - row0);
      float *wo = a.ws_o + slot * D + q4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) *(f32x4 *)(wo + dt * 16) = o[rb][dt];
      if (lane < 16) {
        a.ws_ml[slot * 2 + 0] = m_run[rb];
        a.ws_ml[slot * 2 + 1] = l_tot;
      }
    }
  }
}

// Merges the per-chunk partials of every (request, kv-head, row tile) whose
// prefix was split: out = sum_c 2^(m_c - m) o_c / sum_c 2^(m_c - m) l_c.
template <int D>
__global__ __launch_bounds__(kThreads) void tree_attn_combine_kernel(TreeAttnArgs a) {
  const int64_t gid = blockIdx.x;
  if (gid >= a.row_groups) return;
  int32_t r;
  int64_t ubase, gbase;
  if (!locate_request(gid, true, a, r, ubase, gbase)) return;
  const int32_t node_base = a.node_indptr[r];
  const int32_t n = min(max(a.node_indptr[r + 1] - node_base, 0), kMaxTreeNodes);
  if (n == 0 || node_base < 0 || node_base + n > a.total_nodes) return;
  const int32_t L = max(a.prefix_len[r], 0);
  const int G = a.group;
  const int32_t tiles = row_tiles(n, G);
  const int32_t chunks = prefix_chunks(L, a.chunk_keys);
  if (chunks == 1) return;
  const int64_t u = gid - gbase;
  const int32_t tile = (int32_t)(u % tiles);
  const int32_t g = (int32_t)(u / tiles);
  const int32_t rows = min(kRowsPerTile, n * G - tile * kRowsPerTile);
  constexpr int TPR = D / 4;
  constexpr int RPP = kThreads / TPR;
  const int d4 = (threadIdx.x % TPR) * 4;
  for (int rl = threadIdx.x / TPR; rl < rows; rl += RPP) {
    float mmax = -INFINITY;
    for (int c = 0; c < chunks; ++c) {
      const int64_t unit = ubase + ((int64_t)g * chunks + c) * tiles + tile;
      mmax = fmaxf(mmax, a.ws_ml[(unit * kRowsPerTile + rl) * 2]);
    }
    float den = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < chunks; ++c) {
      const int64_t unit = ubase + ((int64_t)g * chunks + c) * tiles + tile;
      const int64_t slot = unit * kRowsPerTile + rl;
      const float w = __builtin_amdgcn_exp2f(a.ws_ml[slot * 2] - mmax);
      den += w * a.ws_ml[slot * 2 + 1];
      acc += w * *(const f32x4 *)(a.ws_o + slot * D + d4);
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int row = tile * kRowsPerTile + rl;
    const int node = row / G, hh = row - (row / G) * G;
    __bf16 *op = (__bf16 *)a.out + ((int64_t)(node_base + node) * a.num_q_heads + g * G + hh) * D + d4;
    u32x2 w;
    w[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    w[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *(u32x2 *)op = w;
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

hipError_t launch_tree_attn_bf16(const TreeAttnArgs &a, int head_dim, bool needs_combine,
                                 hipStream_t stream) {
  if (a.units == 0) return hipSuccess;
  const dim3 grid((unsigned)a.padded_grid), block(kThreads);
  if (head_dim == 128)
    hipLaunchKernelGGL(tree_attn_bf16_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_attn_bf16_kernel<64>, grid, block, 0, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !needs_combine) return err;
  const dim3 cgrid((unsigned)a.row_groups);
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
