// One beam-search speculation step on gfx950 (section 4.3 step 1).
//
// Every beam node b of a request expands into all |V| tokens; a child's
// path probability is f(b) times the draft model's softmax probability of
// the token, and each request keeps the beam_out children with the highest
// path probability.  In logs: score(b, t) = log f(b) + x[b, t] - lse(x[b, :]).
//
// The logits are the only large operand (beam rows x |V|), so the step is a
// single HBM stream followed by a tiny merge:
//
//  * beam_scan_kernel: a workgroup of 8 waves covers a part of a row; each
//    wave holds one chunk (64 lanes x 16 vectors of 16 bytes) in registers.
//    One pass takes each lane's running maximum and exponential sum.  The
//    chunk's best K = beam_out logits are then found without sorting the
//    chunk: the K-th largest lane maximum T is a lower bound of the K-th
//    largest logit (K lanes hold a value >= T), so every one of the best K
//    is >= T and sits in a "hot" lane (lane maximum >= T).  T comes from a
//    bitwise radix select on ballots (32 steps of one compare and a
//    popcount).  Hot lanes (usually K of them) copy their vectors to LDS,
//    the whole wave filters them against T, and each of the (at most 64)
//    survivors is placed by counting the survivors that beat it.  Many hot
//    lanes or survivors (ties at T, sorted rows, wide beams) take a general
//    path: a threshold-filtered LDS buffer cut back to its K best whenever
//    it could overflow.  The workgroup's list is the K best of its waves'
//    lists, again placed by counting, plus the merged (max, sum).
//  * beam_merge_kernel: one workgroup per request turns the parts' (max,
//    sum) into lse per beam, adds log f(b) - lse to the parts' listed
//    logits (the offset is the same for a whole row, so a row's best
//    children by logit are its best by score), ranks each beam's candidates
//    by counting, and takes the beam_out best of the beams' lists: each
//    placed by counting when they all have a thread, else head by head in
//    beam_out rounds of a wave maximum.
//
// Entries travel as 64-bit keys whose unsigned order is the ranking order
// (see row_key and child_key), so every comparison is one integer compare
// and every cross-lane reduction moves two dwords, on DPP row rotations and
// permlane swaps rather than LDS permutes.  Rows of beams with log f = -inf
// (unused slots) are not read at all.
#include <limits.h>

#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kVecPerLane = 16;       // 16-byte vectors per lane per chunk
constexpr int kScanWaves = 8;         // chunks (waves) per workgroup
constexpr int kGather = 64;           // fast-path candidates per chunk
constexpr int kCap = 640;             // general-path buffer entries per wave
constexpr int kStageLanes = 20;       // hot lanes staged in LDS (kStageLanes x 256 B fit the buffer)
constexpr int kStageRounds = (kStageLanes * kVecPerLane + 63) / 64;
static_assert(kStageLanes * kVecPerLane * 16 <= kCap * 8, "staged vectors must fit the per-wave buffer");
constexpr int kMergeEntries = 4096;   // candidates staged in LDS by the merge
constexpr int kMergeThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Orderable unsigned image of a float: a < b  <=>  key(a) < key(b).
__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Order inside a row: larger logit first, then smaller token.  0 = none
// (below every real entry: even -inf has a nonzero high word).
__device__ __forceinline__ uint64_t row_key(float x, int tok) {
  return ((uint64_t)order_key(x) << 32) | (uint32_t)~tok;
}
__device__ __forceinline__ float row_key_value(uint64_t k) { return key_value((uint32_t)(k >> 32)); }
__device__ __forceinline__ int row_key_token(uint64_t k) { return (int)~(uint32_t)k; }

// Order across a request: higher float32 score, then smaller beam, then
// smaller token (tokens < 2^20, beams < 64).
__device__ __forceinline__ uint64_t child_key(float score, int beam, int tok) {
  return ((uint64_t)order_key(score) << 32) | ((uint32_t)(63 - beam) << 20) | (uint32_t)(0xfffff - tok);
}

// DPP rotation inside each row of 16 lanes: lane i gets lane (i - N) mod 16.
template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x120 + N, 0xf, 0xf, false);
}

template <int N>
__device__ __forceinline__ uint64_t max_ror(uint64_t k) {
  const uint64_t o = ((uint64_t)row_ror<N>((uint32_t)(k >> 32)) << 32) | row_ror<N>((uint32_t)k);
  return o > k ? o : k;
}

// Maximum over the wave, in every lane: rotations inside rows, then the
// permlane swaps that pair rows (16) and halves (32).  Every step is a
// reduction, so the direction of each exchange does not matter.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t k) {
  k = max_ror<8>(k);
  k = max_ror<4>(k);
  k = max_ror<2>(k);
  k = max_ror<1>(k);
  {
    auto h = __builtin_amdgcn_permlane16_swap((uint32_t)(k >> 32), (uint32_t)(k >> 32), false, false);
    auto l = __builtin_amdgcn_permlane16_swap((uint32_t)k, (uint32_t)k, false, false);
    const uint64_t k0 = ((uint64_t)h[0] << 32) | l[0], k1 = ((uint64_t)h[1] << 32) | l[1];
    k = k0 > k1 ? k0 : k1;
  }
  {
    auto h = __builtin_amdgcn_permlane32_swap((uint32_t)(k >> 32), (uint32_t)(k >> 32), false, false);
    auto l = __builtin_amdgcn_permlane32_swap((uint32_t)k, (uint32_t)k, false, false);
    const uint64_t k0 = ((uint64_t)h[0] << 32) | l[0], k1 = ((uint64_t)h[1] << 32) | l[1];
    k = k0 > k1 ? k0 : k1;
  }
  return k;
}

__device__ __forceinline__ float wave_max_f32(float v) {
  return key_value((uint32_t)(wave_max_u64((uint64_t)order_key(v) << 32) >> 32));
}

// K-th largest of the 64 lanes' keys (1 <= K <= 64): the largest t with at
// least K lanes >= t, built bit by bit from ballots.
__device__ __forceinline__ uint32_t kth_largest_key(uint32_t key, int K) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if (__popcll(__ballot(key >= c)) >= K) t = c;
  }
  return t;
}

// Element e of a 16-byte vector, widened exactly to fp32.
template <bool BF16>
__device__ __forceinline__ float elem(const u32x4 &w, int e) {
  if (BF16) return __uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
  return __uint_as_float(w[e]);
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Keeps the `k` best keys of buf[0, count) (the general path).  Keys are
// unique (token ids differ), so "best key below the previous pick" needs no
// marks.  Lane j < kept ends with key j in `out`, the rest with 0; the kept
// keys are also written back to buf[0, kept).
__device__ int keep_best(uint64_t *buf, int count, int k, uint64_t &out) {
  const int lane = threadIdx.x & 63;
  uint64_t prev = ~0ull;
  int kept = 0;
  out = 0;
  for (int r = 0; r < k; ++r) {
    uint64_t c = 0;
    for (int j = lane; j < count; j += 64) {
      const uint64_t e = buf[j];
      if (e < prev && e > c) c = e;
    }
    c = wave_max_u64(c);
    if (c == 0) break;  // no entry left
    if (lane == r) out = c;
    prev = c;
    ++kept;
  }
  wave_sync_lds();
  if (lane < kept) buf[lane] = out;
  wave_sync_lds();
  return kept;
}

// Writes the K best of cand[0, n) (n <= 64, unique keys) to out[0, K) in
// order, 0 past the n-th: each lane ranks one candidate by counting the
// candidates that beat it.
__device__ __forceinline__ void rank_into(const uint64_t *cand, int n, int K, uint64_t *out) {
  const int lane = threadIdx.x & 63;
  const uint64_t c = lane < n ? cand[lane] : 0;
  int rank = 0;
#pragma unroll 8
  for (int j = 0; j < n; ++j) rank += cand[j] > c;
  if (lane < n && rank < K) out[rank] = c;
  if (lane >= n && lane < K) out[lane] = 0;
}

template <bool BF16>
__global__ __launch_bounds__(64 * kScanWaves) void beam_scan_kernel(BeamArgs a) {
  constexpr int EPV = BF16 ? 8 : 4;
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int kChunk = 64 * kVecPerLane * EPV;
  __shared__ __attribute__((aligned(16))) uint64_t buf[kScanWaves][kCap];
  __shared__ uint64_t lst[kScanWaves * kBeamMaxWidth];  // wave w's sorted list at [w * K, w * K + K)
  __shared__ uint64_t cand[kScanWaves][kGather];
  __shared__ int stage_lane[kScanWaves][kStageLanes];
  __shared__ int gathered[kScanWaves];
  __shared__ float wave_m[kScanWaves], wave_s[kScanWaves];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int row = blockIdx.x / a.parts;
  const int part = blockIdx.x - row * a.parts;
  const int K = a.beam_out;
  const int first = (part * kScanWaves + wave) * kChunk;  // token id of the chunk's first logit
  uint64_t *bw = buf[wave];

  // Running (max, sum of exp(x - max)) of the lane, and the wave's sorted
  // list (lane j holds its j-th best key; 0 past the end).
  float lane_m = -INFINITY, lane_s = 0.f;
  uint64_t mine = 0;
  const bool live = a.beam_logprob[row] > -INFINITY;  // unused slot (or NaN): not read
  if (live && first < a.vocab) {
    const int n_valid = min(kChunk, a.vocab - first);
    const char *base = (const char *)a.logits + ((int64_t)row * a.row_stride + first) * ESZ;
    const uint32_t neg_inf_bits = BF16 ? 0xff80ff80u : 0xff800000u;
    // Whole chunks (every chunk but a row's last) load in straight-line code
    // and the pass follows in the same branch, so it starts on the first
    // vector while the others are still in flight (where the loads sit under
    // branches, or the two ways join before the pass, the compiler waits for
    // all of them first).
    u32x4 w[kVecPerLane];
    float vmax[kVecPerLane];
    auto load_and_pass = [&](auto whole_chunk) {
      if constexpr (decltype(whole_chunk)::value) {
#pragma unroll
        for (int v = 0; v < kVecPerLane; ++v)
          w[v] = __builtin_nontemporal_load((const u32x4 *)(base + (int64_t)(v * 64 + lane) * EPV * ESZ));
      } else {
#pragma unroll
        for (int v = 0; v < kVecPerLane; ++v) {
          const int e0 = (v * 64 + lane) * EPV;
          if (e0 + EPV <= n_valid) {
            w[v] = __builtin_nontemporal_load((const u32x4 *)(base + (int64_t)e0 * ESZ));
          } else {
            u32x4 t = {neg_inf_bits, neg_inf_bits, neg_inf_bits, neg_inf_bits};
            for (int e = 0; e < EPV && e0 + e < n_valid; ++e) {
              if (BF16) {
                const uint32_t h = ((const uint16_t *)base)[e0 + e];
                t[e >> 1] = (e & 1) ? ((t[e >> 1] & 0xffffu) | (h << 16)) : ((t[e >> 1] & 0xffff0000u) | h);
              } else {
                t[e] = ((const uint32_t *)base)[e0 + e];
              }
            }
            w[v] = t;
          }
        }
      }
      // One pass: per-vector maxima, running lane maximum and sum.
#pragma unroll
      for (int v = 0; v < kVecPerLane; ++v) {
        float m = elem<BF16>(w[v], 0);
#pragma unroll
        for (int e = 1; e < EPV; ++e) m = fmaxf(m, elem<BF16>(w[v], e));
        vmax[v] = m;
        const float nm = fmaxf(lane_m, m);
        if (nm > -INFINITY) {
          const float off = -nm * kLog2e;
          float add = 0.f;
#pragma unroll
          for (int e = 0; e < EPV; ++e) add += __builtin_amdgcn_exp2f(fmaf(elem<BF16>(w[v], e), kLog2e, off));
          lane_s = fmaf(lane_s, __builtin_amdgcn_exp2f(fmaf(lane_m, kLog2e, off)), add);
          lane_m = nm;
        }
      }
    };
    if (n_valid == kChunk)
      load_and_pass(std::true_type{});
    else
      load_and_pass(std::false_type{});
    // The widened values are recomputed below rather than kept live.
#pragma unroll
    for (int v = 0; v < kVecPerLane; ++v) asm volatile("" : "+v"(w[v]));

    // Threshold: the K-th largest lane maximum.  Only "hot" lanes (maximum
    // >= T) hold logits >= T; they copy their vectors to LDS, where the whole
    // wave filters them.
    const float T = key_value(kth_largest_key(order_key(lane_m), K));
    const bool hot = lane_m >= T && lane_m > -INFINITY;
    const uint64_t hot_mask = __ballot(hot);
    const int n_hot = __popcll(hot_mask);
    int n_cand = kGather + 1;
    if (n_hot <= kStageLanes) {
      u32x4 *st = (u32x4 *)bw;
      if (lane == 0) gathered[wave] = 0;
      if (hot) {
        const int slot = __popcll(hot_mask & ((1ull << lane) - 1));
#pragma unroll
        for (int v = 0; v < kVecPerLane; ++v) st[slot * kVecPerLane + v] = w[v];
        stage_lane[wave][slot] = lane;
      }
      wave_sync_lds();
      const int n_vec = n_hot * kVecPerLane;
      u32x4 sv[kStageRounds];
      int n = 0;
#pragma unroll
      for (int i = 0; i < kStageRounds; ++i) {
        const int q = lane + 64 * i;
        if (q < n_vec) {
          sv[i] = st[q];
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            const float x = elem<BF16>(sv[i], e);
            n += (x >= T && x > -INFINITY);
          }
        }
      }
      int slot = n ? atomicAdd(&gathered[wave], n) : 0;
#pragma unroll
      for (int i = 0; i < kStageRounds; ++i) {
        const int q = lane + 64 * i;
        if (q < n_vec) {
          const int tok0 = first + ((q % kVecPerLane) * 64 + stage_lane[wave][q / kVecPerLane]) * EPV;
#pragma unroll
          for (int e = 0; e < EPV; ++e) {
            const float x = elem<BF16>(sv[i], e);
            if (x >= T && x > -INFINITY) {
              if (slot < kGather) cand[wave][slot] = row_key(x, tok0 + e);
              ++slot;
            }
          }
        }
      }
      wave_sync_lds();
      n_cand = gathered[wave];
      if (n_cand <= kGather) rank_into(cand[wave], n_cand, K, lst + wave * K);
    }
    if (n_cand > kGather) {
      // General path (ties at T, sorted rows, wide beams): filter against a
      // rising threshold key; keys not below it are buffered, and the buffer
      // is cut back to its K best before it could overflow.  Starts at the
      // smallest key of value T.
      uint64_t thr = (uint64_t)order_key(T) << 32;
      int count = 0;
      wave_sync_lds();
#pragma unroll
      for (int v = 0; v < kVecPerLane; ++v) {
        if (!__any(vmax[v] >= key_value((uint32_t)(thr >> 32)) && vmax[v] > -INFINITY)) continue;
        if (count + 64 * EPV > kCap) {
          count = keep_best(bw, count, K, mine);
          if (count == K) {
            const uint64_t t = (uint64_t)__shfl((unsigned long long)mine, K - 1, 64);
            thr = t;
          }
        }
        const int e0 = first + (v * 64 + lane) * EPV;
        int n = 0;
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
          const float x = elem<BF16>(w[v], e);
          n += (x > -INFINITY && row_key(x, e0 + e) >= thr);
        }
        int incl = n;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int o = __shfl_up(incl, off, 64);
          if (lane >= off) incl += o;
        }
        int j = count + incl - n;
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
          const float x = elem<BF16>(w[v], e);
          const uint64_t key = row_key(x, e0 + e);
          if (x > -INFINITY && key >= thr) bw[j++] = key;
        }
        count += __shfl(incl, 63, 64);
        wave_sync_lds();
      }
      if (count <= kGather) {
        rank_into(bw, count, K, lst + wave * K);
      } else {
        keep_best(bw, count, K, mine);
        if (lane < K) lst[wave * K + lane] = mine;
      }
    }
  } else if (lane < K) {  // unused beam slot, or a chunk past the vocabulary
    lst[wave * K + lane] = 0;
  }

  // The workgroup's (max, sum) and its best K over the waves' lists, each
  // list entry ranked against all of them.
  const float M = wave_max_f32(lane_m);
  float s = M > -INFINITY && lane_m > -INFINITY ? lane_s * __builtin_amdgcn_exp2f((lane_m - M) * kLog2e) : 0.f;
  s = wave_sum(s);
  if (lane == 0) {
    wave_m[wave] = M;
    wave_s[wave] = s;
  }
  __syncthreads();
  const int64_t unit = blockIdx.x;
  const int t = threadIdx.x;
  const int n = kScanWaves * K;
  if (t < n) {
    const uint64_t c = lst[t];
    int rank = 0, nz = 0;
#pragma unroll 8
    for (int j = 0; j < n; ++j) {
      const uint64_t e = lst[j];
      rank += e > c;
      nz += e != 0;
    }
    uint64_t *top = a.ws_top + unit * K;
    if (c != 0 && rank < K) top[rank] = c;
    if (t < K && t >= nz) top[t] = 0;
  }
  if (t == 0) {
    float pm = -INFINITY;
    for (int w = 0; w < kScanWaves; ++w) pm = fmaxf(pm, wave_m[w]);
    float ps = 0.f;
    if (pm > -INFINITY)
      for (int w = 0; w < kScanWaves; ++w)
        if (wave_m[w] > -INFINITY) ps += wave_s[w] * __builtin_amdgcn_exp2f((wave_m[w] - pm) * kLog2e);
    a.ws_ml[unit] = make_float2(pm, ps);
  }
}

__global__ __launch_bounds__(kMergeThreads) void beam_merge_kernel(BeamArgs a) {
  __shared__ float offset[kBeamMaxWidth];
  __shared__ uint64_t cand[kMergeEntries];                      // child keys of a batch of beams
  __shared__ uint64_t blist[kBeamMaxWidth * kBeamMaxWidth];     // beam b's sorted list at [b * K, b * K + K)
  const int r = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63;
  const int W = a.beam_in, P = a.parts, K = a.beam_out;
  const int per_beam = P * K;
  const uint64_t *top = a.ws_top + (int64_t)r * W * per_beam;

  // log f(b) - lse(row b) per beam, from the row's parts.
  for (int b = t; b < W; b += kMergeThreads) {
    const int row = r * W + b;
    const float2 *ml = a.ws_ml + (int64_t)row * P;
    float m = -INFINITY;
    for (int p = 0; p < P; ++p) m = fmaxf(m, ml[p].x);
    float s = 0.f;
    if (m > -INFINITY)
      for (int p = 0; p < P; ++p)
        if (ml[p].x > -INFINITY) s += ml[p].y * exp2f((ml[p].x - m) * kLog2e);
    const float lp = a.beam_logprob[row];
    offset[b] = (lp > -INFINITY && m > -INFINITY) ? lp - (m + log2f(s) * kLn2) : -INFINITY;
  }
  __syncthreads();

  // Each beam's best K children, ranked among its parts' lists, in batches
  // of beams whose candidates fit in LDS.
  const int batch = kMergeEntries / per_beam;  // >= 1: per_beam <= kBeamMaxParts * kBeamMaxWidth
  for (int b0 = 0; b0 < W; b0 += batch) {
    const int n = min(batch, W - b0) * per_beam;
    for (int c = t; c < n; c += kMergeThreads) {
      const int b = b0 + c / per_beam;
      const uint64_t e = top[(int64_t)b0 * per_beam + c];
      uint64_t key = 0;
      if (e != 0) {
        const float x = row_key_value(e);
        const float score = offset[b] + x;
        if (x > -INFINITY && score > -INFINITY) key = child_key(score, b, row_key_token(e));
      }
      cand[c] = key;
    }
    __syncthreads();
    for (int c = t; c < n; c += kMergeThreads) {
      const int base = c / per_beam * per_beam;
      const uint64_t key = cand[c];
      int rank = 0, nz = 0;
#pragma unroll 8
      for (int j = 0; j < per_beam; ++j) {
        const uint64_t e = cand[base + j];
        rank += e > key;
        nz += e != 0;
      }
      const int b = b0 + c / per_beam;
      if (key != 0 && rank < K) blist[b * K + rank] = key;
      const int pos = c - base;
      if (pos < K && pos >= nz) blist[b * K + pos] = 0;
    }
    __syncthreads();
  }

  // The beam_out best of the W·K listed children.  When every one of them
  // has a thread, each is placed by counting the larger keys (keys are
  // unique; 0 = no child); otherwise a head merge across the beams' sorted
  // lists, lane b following beam b, takes the best head beam_out times.
  if (W * K <= kMergeThreads) {
    const int all = W * K;
    const uint64_t c = t < all ? blist[t] : 0;
    int rank = 0, nz = 0;
    if (t < all) {
#pragma unroll 8
      for (int j = 0; j < all; ++j) {
        const uint64_t e = blist[j];
        rank += e > c;
        nz += e != 0;
      }
    }
    if (c != 0 && rank < K) {
      a.out_parent[r * K + rank] = 63 - (int)((c >> 20) & 63);
      a.out_token[r * K + rank] = 0xfffff - (int)(c & 0xfffff);
      a.out_logprob[r * K + rank] = key_value((uint32_t)(c >> 32));
    }
    if (t < K && t >= nz) {  // fewer children than slots (t < K <= all, so nz is this thread's count)
      a.out_parent[r * K + t] = -1;
      a.out_token[r * K + t] = -1;
      a.out_logprob[r * K + t] = -INFINITY;
    }
    return;
  }
  if (t >= 64) return;
  int head = 0;
  uint64_t cur = lane < W ? blist[lane * K] : 0;
  int k = 0;
  for (; k < K; ++k) {
    const uint64_t m = wave_max_u64(cur);
    if (m == 0) break;  // fewer children than slots
    if (lane == 0) {
      a.out_parent[r * K + k] = 63 - (int)((m >> 20) & 63);
      a.out_token[r * K + k] = 0xfffff - (int)(m & 0xfffff);
      a.out_logprob[r * K + k] = key_value((uint32_t)(m >> 32));
    }
    if (lane < W && cur == m) {
      ++head;
      cur = head < K ? blist[lane * K + head] : 0;
    }
  }
  for (int j = k + lane; j < K; j += 64) {
    a.out_parent[r * K + j] = -1;
    a.out_token[r * K + j] = -1;
    a.out_logprob[r * K + j] = -INFINITY;
  }
}

}  // namespace

int32_t beam_parts(int32_t vocab, bool bf16) {
  const int64_t per_part = (int64_t)kScanWaves * 64 * kVecPerLane * (bf16 ? 8 : 4);
  return (int32_t)((vocab + per_part - 1) / per_part);
}

hipError_t launch_beam_step(const BeamArgs &a, bool bf16, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((int64_t)a.rows * a.parts);
  if (bf16)
    hipLaunchKernelGGL(beam_scan_kernel<true>, dim3(blocks), dim3(64 * kScanWaves), 0, stream, a);
  else
    hipLaunchKernelGGL(beam_scan_kernel<false>, dim3(blocks), dim3(64 * kScanWaves), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(beam_merge_kernel, dim3((unsigned)a.num_requests), dim3(kMergeThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
