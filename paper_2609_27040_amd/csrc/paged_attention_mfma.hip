// Paged decode attention on the matrix cores (gfx950 MFMA 16x16x32).
//
// With grouped-query attention the G query heads that share a KV head turn
// decode into a small dense contraction per KV head: [G x 128] . [128 x T] for
// the scores and [G x T] . [T x 128] for the output. Both go to
// v_mfma_f32_16x16x32_{bf16,f16} (G <= 16 heads fill one 16-wide tile), which
// leaves the vector ALUs nearly idle and the kernel bound by HBM.
//
// Work is cut into 32-token tiles of one (sequence, KV head). Each wavefront
// streams tiles with an online softmax, two tiles in flight:
//   scores   S^T[token][head] = K . Q^T   (A = 16 K rows straight from the
//            block, B = Q^T held in registers; two 16-token tiles whose rows
//            are chosen so that each lane ends up holding 8 consecutive
//            tokens of one head -- exactly the B-operand layout of the next
//            product, so no data moves between lanes)
//   output   O^T[channel][head] += V^T . P^T  (A = 16 channel rows of the
//            transposed V block, 8 consecutive tokens per lane, 16 B loads;
//            P is split into a 16-bit high part and a 16-bit remainder so the
//            probabilities keep ~16 significant bits)
// Scheduling is stream-K: the tiles of all (sequence, KV head) pairs, in that
// order, are split into equal contiguous ranges, one per workgroup of 4
// wavefronts and one workgroup per CU, so every CU streams the same bytes
// whatever the length mix. A workgroup keeps its softmax state across the
// tiles of one (sequence, KV head) and issues the first loads of its next
// pair before merging the current one; a pair it covers whole is written out
// directly, a pair cut by a range boundary leaves one partial per workgroup
// (unnormalised output, max, sum) that a small combine kernel merges. Merging
// inside this kernel costs more: partials must cross XCDs, whose L2s are not
// coherent, either behind device-scope fences (a whole-L2 write-back and
// invalidation per workgroup) or as written-through stores plus an arrival
// counter, and either way at the end of every workgroup's range. Masked tokens
// (past the length, or in a block whose id is out of range) get -inf scores
// and zeroed V, so NaN in unused slots never leaks.
// Reduction orders depend only on sequence lengths, not on block ids.
#include "attn_store.h"
#include "kernels.h"

#include <algorithm>
#include <cmath>
#include <mutex>
#include <unordered_map>

namespace ema {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kIt = 32;                    // tokens per tile (one wave iteration)
constexpr int kPieceTiles = 32;            // tiles whose block ids are staged in LDS at once
constexpr int kMaxIds = kPieceTiles * kIt / 16;
constexpr int kGridChunkTiles = 32;        // tiles per workgroup in the grid fallback
// Each (sequence, KV head) a workgroup touches costs it several tiles' time
// (the four wavefronts merge and a partial is written; without the staged
// range below, the tile pipeline also drains and refills); the stream-K split
// counts it as seg_cost<G>() tiles so that workgroups that touch more pairs
// get fewer tiles. Measured on 32-token tiles with one workgroup per CU: 8 is
// best between 6 and 10 at 4 and 8 query heads per KV head; 16 query heads,
// whose merge and partials are four times larger, do best with 16 (against
// 8, 12 and 24).
template <int G>
constexpr int seg_cost() { return G >= 16 ? 16 : 8; }
// A stream-K range whose segments and block ids fit these bounds is staged
// in LDS up front, so each segment can start while the previous one merges.
constexpr int kMaxSegMax = 8;              // segments of a range (4 for G = 16)
template <int G>
constexpr int max_seg() { return G >= 16 ? 4 : kMaxSegMax; }
constexpr int kRangeIds = 512;             // block ids of a range

__device__ __forceinline__ u32x4 ld16(const char* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
// K/V are read exactly once per call: streaming loads keep them from
// displacing tables, queries and partials in L2 and the memory-side cache.
__device__ __forceinline__ u32x4 ld16_stream(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <bool BF16>
__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// p -> (high, low) 16-bit parts with p ~= high + low.
template <bool BF16>
__device__ __forceinline__ void split16(float p, uint32_t& hi, uint32_t& lo) {
  if constexpr (BF16) {
    const uint32_t u = __builtin_bit_cast(uint32_t, p);
    hi = u >> 16;                                        // truncation: exact remainder
    const float r = p - __builtin_bit_cast(float, u & 0xffff0000u);
    const uint32_t v = __builtin_bit_cast(uint32_t, r);
    lo = (v + 0x7fffu + ((v >> 16) & 1u)) >> 16;         // round to nearest even
  } else {
    const _Float16 h = _Float16(p);
    const _Float16 l = _Float16(p - float(h));
    hi = __builtin_bit_cast(uint16_t, h);
    lo = __builtin_bit_cast(uint16_t, l);
  }
}

__device__ __forceinline__ int clamp_len(int len, const AttnArgs& a) {
  const int cap = a.max_blocks * a.block_size;
  return len < 0 ? 0 : (len > cap ? cap : len);
}

// One 32-token iteration's operands: K rows of the two score tiles and the
// eight V^T row tiles, plus how many of this lane's 8 tokens are valid.
struct Tile {
  u32x4 k[2][4];
  u32x4 v[8];
  int nv;
};

// Issues the loads of the tile starting at token t0 of the sequence. Every lane
// loads unconditionally (a lane whose token is masked reads block 0, which
// always exists), so the loads stay in straight-line code and the compiler can
// wait for this tile alone while the next one is in flight. K rows of masked
// tokens only reach scores that consume_tile sets to -inf; V of masked tokens
// is zeroed there before use.
template <int BS>
__device__ __forceinline__ void load_tile(Tile& T, int t0, int len, int blk0, const int32_t* s_ids,
                                          const char* pool, int64_t Bb, int kvh, int r16,
                                          int q4) {
  // K rows: tile t, row r16 -> token t0 + 8*(r16/4) + 4t + r16%4.
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tok = t0 + 8 * (r16 >> 2) + 4 * t + (r16 & 3);
    const int id = s_ids[tok / BS - blk0];
    const bool ok = tok < len && id >= 0;
    const char* p = pool + (ok ? int64_t(id) * Bb + (int64_t(kvh * BS + tok % BS) * kD + q4 * 8) * 2
                               : int64_t(0));
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) T.k[t][kk] = ld16_stream(p + kk * 64);
  }
  // V^T rows: d-tile n, row 16n + r16, tokens t0 + 8q4 .. +8 (one block).
  const int vt = t0 + 8 * q4;
  const int vid = s_ids[vt / BS - blk0];
  const int vleft = len - vt;
  T.nv = vid < 0 ? 0 : (vleft < 0 ? 0 : (vleft > 8 ? 8 : vleft));
  const char* p = pool + (T.nv > 0 ? int64_t(vid) * Bb + Bb / 2 +
                                         (int64_t(kvh * kD + r16) * BS + vt % BS) * 2
                                   : int64_t(0));
#pragma unroll
  for (int n = 0; n < 8; ++n) T.v[n] = ld16_stream(p + int64_t(16 * n) * BS * 2);
}

// Scores, online softmax update and P.V for one loaded iteration.
// `issue_next` runs right after the score products are issued: loads of the
// next tile then queue behind this tile's V loads, so the in-order wait
// before P.V covers this tile only.
template <bool BF16, typename Next>
__device__ __forceinline__ void consume_tile(Tile& T, const u32x4 (&qb)[4], float scale_log2,
                                             float& m, float& lsum, f32x4 (&o)[8],
                                             Next&& issue_next) {
  const int nv = T.nv;
#pragma unroll
  for (int q = 0; q < 4; ++q) {   // branch-free, so waits stay per tile
    const uint32_t keep = (2 * q < nv ? 0xffffu : 0u) | (2 * q + 1 < nv ? 0xffff0000u : 0u);
#pragma unroll
    for (int n = 0; n < 8; ++n) T.v[n][q] &= keep;
  }
  // Scores for tokens 8q4 + 4t + i of head r16.
  f32x4 s[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    s[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) s[t] = mfma<BF16>(T.k[t][kk], qb[kk], s[t]);
  }
  issue_next();
  float sv[8];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    sv[j] = j < nv ? s[j >> 2][j & 3] * scale_log2 : -INFINITY;
    mx = fmaxf(mx, sv[j]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(m, mx);
  const float alpha = m_new == -INFINITY ? 1.0f : exp2f(m - m_new);
  uint32_t ph[4], pl[4];
  float ps = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float p0 = m_new == -INFINITY ? 0.0f : exp2f(sv[2 * q] - m_new);
    const float p1 = m_new == -INFINITY ? 0.0f : exp2f(sv[2 * q + 1] - m_new);
    ps += p0 + p1;
    uint32_t h0, l0, h1, l1;
    split16<BF16>(p0, h0, l0);
    split16<BF16>(p1, h1, l1);
    ph[q] = h0 | (h1 << 16);
    pl[q] = l0 | (l1 << 16);
  }
  lsum = lsum * alpha + ps;
  m = m_new;
  const u32x4 PH = {ph[0], ph[1], ph[2], ph[3]};
  const u32x4 PL = {pl[0], pl[1], pl[2], pl[3]};
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    o[n] *= alpha;
    o[n] = mfma<BF16>(T.v[n], PH, o[n]);
    o[n] = mfma<BF16>(T.v[n], PL, o[n]);
  }
}

template <int G>
struct Smem {
  int32_t ids[kMaxIds];
  __attribute__((aligned(16))) float o[kWaves][G][kD];
  float m[kWaves][G];
  float l[kWaves][G];
};

// Attends tiles [j0, j1) of (sequence b, KV head kvh) with all four waves
// (wave w takes tiles j0 + w, j0 + w + 4, ...; two tiles in flight) and hands
// the merged (max, sum, unnormalised output) of each (head g, channel d) to
// emit(), with the (g, d) pairs spread over the workgroup's threads.
template <int G, int BS, bool BF16, typename Emit>
__device__ __forceinline__ void attend_segment(const AttnArgs& a, int b, int kvh, int len, int j0,
                                               int j1, Smem<G>& sm, Emit&& emit) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;
  const int q4 = lane >> 4;
  // Q^T as the B operand: lane (head r16, q4) holds channels 32kk + 8q4 .. +8.
  u32x4 qb[4];
  {
    const char* qrow = reinterpret_cast<const char*>(a.q) +
                       (int64_t(b) * a.q_heads + kvh * G + r16) * kD * 2 + q4 * 16;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      qb[kk] = r16 < G ? ld16(qrow + kk * 64) : u32x4{0, 0, 0, 0};
  }
  const char* pool = a.local;
  const int64_t Bb = a.block_bytes;
  float m = -INFINITY;   // running max of this lane's head (log2 domain)
  float lsum = 0.0f;     // this lane's share of the running sum
  f32x4 o[8];
#pragma unroll
  for (int n = 0; n < 8; ++n) o[n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  for (int p0 = j0; p0 < j1; p0 += kPieceTiles) {
    const int p1 = min(j1, p0 + kPieceTiles);
    const int blk0 = p0 * kIt / BS;
    const int cnt = (p1 * kIt - 1) / BS - blk0 + 1;
    __syncthreads();                      // the previous piece's ids are no longer read
    if (tid < cnt) {
      const int j = blk0 + tid;
      int id = -1;
      if (j * BS < len) {
        id = a.table[int64_t(b) * a.max_blocks + j];
        if (id < 0 || id >= a.n_local) {
          atomicAdd(a.err_count, 1);
          id = -1;
        }
      }
      sm.ids[tid] = id;
    }
    __syncthreads();
    const int nt = p1 - p0;
    const int n_it = nt > wave ? (nt - wave + kWaves - 1) / kWaves : 0;
    auto load_at = [&](Tile& T, int k) {
      load_tile<BS>(T, (p0 + wave + k * kWaves) * kIt, len, blk0, sm.ids, pool, Bb, kvh, r16, q4);
    };
    Tile A, B;
    if (n_it > 0) load_at(A, 0);
    for (int it = 0; it < n_it; it += 2) {
      consume_tile<BF16>(A, qb, a.scale_log2, m, lsum, o, [&] {
        if (it + 1 < n_it) load_at(B, it + 1);
      });
      if (it + 1 >= n_it) break;
      consume_tile<BF16>(B, qb, a.scale_log2, m, lsum, o, [&] {
        if (it + 2 < n_it) load_at(A, it + 2);
      });
    }
  }

  // ---- merge the four waves ------------------------------------------------
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (r16 < G) {
    if (q4 == 0) {
      sm.m[wave][r16] = m;
      sm.l[wave][r16] = lsum;
    }
#pragma unroll
    for (int n = 0; n < 8; ++n)
      *reinterpret_cast<f32x4*>(&sm.o[wave][r16][16 * n + 4 * q4]) = o[n];
  }
  __syncthreads();
  for (int e = tid; e < G * kD; e += kThreads) {
    const int g = e / kD;
    const int d = e % kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.m[w][g]);
    float L = 0.0f, O = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = sm.m[w][g];
        if (mw == -INFINITY) continue;
        const float f = exp2f(mw - M);
        L = fmaf(f, sm.l[w][g], L);
        O = fmaf(f, sm.o[w][g][d], O);
      }
    }
    emit(g, d, M, L, O);
  }
}

// Workgroup-uniform value kept in a scalar register.
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// One segment of a stream-K range: tiles [j0, j1) of (sequence b, KV head
// kvh); id0 is the index of its first block id in the range's staged list.
struct SegDesc {
  int b, kvh, len, j0, j1, id0;
};

// Q^T of segment s from its LDS copy (rows past G read as zero).
template <int G>
__device__ __forceinline__ void load_q(u32x4 (&qb)[4], const uint16_t (*sq)[G][kD], int s, int r16,
                                       int q4) {
  const uint16_t* row = sq[s][r16 < G ? r16 : 0] + q4 * 8;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(row + kk * 32);
    qb[kk] = r16 < G ? v : u32x4{0, 0, 0, 0};
  }
}

// All segments of a stream-K range with their block ids already in LDS: the
// four waves stream tiles as in attend_segment, and each wave issues the loads
// of its first tile of the next segment (and the next segment's queries)
// before the merge of the current one, so no segment starts from an empty
// pipeline.
template <int G, int BS, bool BF16, typename Emit>
__device__ __forceinline__ void attend_range(const AttnArgs& a, const SegDesc* sd, int nseg,
                                             const int32_t* ids, const uint16_t (*sq)[G][kD],
                                             Smem<G>& sm, Emit&& emit) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;
  const int q4 = lane >> 4;
  const char* pool = a.local;
  const int64_t Bb = a.block_bytes;
  auto n_tiles = [&](int s) {
    const int nt = sd[s].j1 - sd[s].j0;
    return nt > wave ? (nt - wave + kWaves - 1) / kWaves : 0;
  };
  auto load_at = [&](Tile& T, int s, int k) {
    const int j0 = uniform(sd[s].j0);
    load_tile<BS>(T, (j0 + wave + k * kWaves) * kIt, uniform(sd[s].len), j0 * kIt / BS,
                  ids + uniform(sd[s].id0), pool, Bb, uniform(sd[s].kvh), r16, q4);
  };
  u32x4 qb[4];
  Tile A, B;
  if (nseg > 0) {
    load_q<G>(qb, sq, 0, r16, q4);
    if (n_tiles(0) > 0) load_at(A, 0, 0);
  }
  for (int s = 0; s < nseg; ++s) {
    const int n_it = n_tiles(s);
    const bool has_next = s + 1 < nseg && n_tiles(s + 1) > 0;
    bool issued_next = false;
    float m = -INFINITY;
    float lsum = 0.0f;
    f32x4 o[8];
#pragma unroll
    for (int n = 0; n < 8; ++n) o[n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int it = 0; it < n_it; it += 2) {
      consume_tile<BF16>(A, qb, a.scale_log2, m, lsum, o, [&] {
        if (it + 1 < n_it) load_at(B, s, it + 1);
      });
      if (it + 1 >= n_it) break;
      consume_tile<BF16>(B, qb, a.scale_log2, m, lsum, o, [&] {
        if (it + 2 < n_it) {
          load_at(A, s, it + 2);
        } else if (has_next) {
          load_at(A, s + 1, 0);
          issued_next = true;
        }
      });
    }
    if (has_next && !issued_next) load_at(A, s + 1, 0);
    if (s + 1 < nseg) load_q<G>(qb, sq, s + 1, r16, q4);

    // ---- merge the four waves (as in attend_segment) ----
    __syncthreads();                       // the previous merge is read out
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    if (r16 < G) {
      if (q4 == 0) {
        sm.m[wave][r16] = m;
        sm.l[wave][r16] = lsum;
      }
#pragma unroll
      for (int n = 0; n < 8; ++n)
        *reinterpret_cast<f32x4*>(&sm.o[wave][r16][16 * n + 4 * q4]) = o[n];
    }
    __syncthreads();
    for (int e = tid; e < G * kD; e += kThreads) {
      const int g = e / kD;
      const int d = e % kD;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.m[w][g]);
      float L = 0.0f, O = 0.0f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
          const float mw = sm.m[w][g];
          if (mw == -INFINITY) continue;
          const float f = exp2f(mw - M);
          L = fmaf(f, sm.l[w][g], L);
          O = fmaf(f, sm.o[w][g][d], O);
        }
      }
      emit(s, g, d, M, L, O);
    }
  }
}

__device__ __forceinline__ void write_zeros(const AttnArgs& a, int b) {
  for (int e = threadIdx.x; e < a.q_heads * kD; e += kThreads)
    store_out(a, int64_t(b) * a.q_heads * kD + e, 0.0f);
}

// Stream-K form. Every workgroup reads all lengths once and prefix-sums the
// unit counts (n_t(b) + kSegCost) * Hkv in LDS (kSegCost = seg_cost<G>());
// units are ordered (sequence, KV head, unit), each pair's kSegCost cost
// units (no tiles) ahead of its n_t tiles, and workgroup w takes units
// [w*per, (w+1)*per), per = ceil(U/grid).
// For each (sequence, KV head) it touches, it writes the output directly when
// it holds all of that pair's tiles, else a partial into slot 2w (its first
// pair) or 2w+1 (its last pair). The workgroup that holds a pair's first tile
// records (first workgroup, last workgroup, its slot) for the combine. When
// the range's segments and block ids fit in LDS (kMaxSegMax, kRangeIds), they
// and the segments' queries are staged once and attend_range carries the
// tile pipeline across segments; otherwise each segment runs on its own.
template <int G, int BS, bool BF16>
// Compiled as if two workgroups shared a CU (at most 256 registers a lane),
// although one per CU is launched: under the looser bound the compiler's
// schedule (which then also used accumulation registers) ran every call
// 11-12 % slower.
__global__ __launch_bounds__(kThreads, 2) void attn_mfma_streamk(AttnArgs a) {
  constexpr int kSegCost = seg_cost<G>();
  __shared__ Smem<G> sm;
  __shared__ int32_t s_len[streamk_max_batch(G)];
  __shared__ int32_t s_pref[streamk_max_batch(G) + 1];
  __shared__ int32_t s_seg[kThreads];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int B = a.batch;
  const int H = a.kv_heads;
  const int per_t = (B + kThreads - 1) / kThreads;
  const int b0 = min(B, tid * per_t);
  const int b1 = min(B, b0 + per_t);
  int run = 0;
  for (int b = b0; b < b1; ++b) {
    const int raw = a.seq_lens[b];
    const int len = clamp_len(raw, a);
    if (blockIdx.x == 0 && len != raw && raw > 0) atomicAdd(a.err_count, 1);
    s_len[b] = len;
    s_pref[b] = run;
    const int nt_b = (len + kIt - 1) / kIt;
    run += nt_b > 0 ? (nt_b + kSegCost) * H : 0;
  }
  s_seg[tid] = run;
  __syncthreads();
  if (tid < 64) {   // exclusive scan of the 256 per-thread totals
    const int v0 = s_seg[4 * lane], v1 = s_seg[4 * lane + 1];
    const int v2 = s_seg[4 * lane + 2], v3 = s_seg[4 * lane + 3];
    int sum = v0 + v1 + v2 + v3;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(sum, o);
      if (lane >= o) sum += t;
    }
    const int ex = sum - (v0 + v1 + v2 + v3);
    s_seg[4 * lane] = ex;
    s_seg[4 * lane + 1] = ex + v0;
    s_seg[4 * lane + 2] = ex + v0 + v1;
    s_seg[4 * lane + 3] = ex + v0 + v1 + v2;
    if (lane == 63) s_pref[B] = sum;
  }
  __syncthreads();
  for (int b = b0; b < b1; ++b) s_pref[b] += s_seg[tid];
  __syncthreads();
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    if (s_len[b] != 0) continue;
    write_zeros(a, b);
    for (int h = tid; h < H; h += kThreads) {
      int32_t* info = a.info + (int64_t(b) * H + h) * 3;
      info[0] = info[1] = info[2] = 0;
    }
  }

  const int U = s_pref[B];
  const int per = (U + int(gridDim.x) - 1) / int(gridDim.x);
  int u = min(U, int(blockIdx.x) * per);
  const int u_end = min(U, u + per);

  // The range's segments and all their block ids, staged once.
  constexpr int kMaxSeg = max_seg<G>();
  __shared__ SegDesc s_desc[kMaxSeg];
  __shared__ int32_t s_rids[kRangeIds];
  __shared__ __attribute__((aligned(16))) uint16_t s_q[kMaxSeg][G][kD];
  int nseg = 0, nids = 0;
  {
    int uu = u;
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_pref[mid] <= uu) lo = mid;
      else hi = mid - 1;
    }
    int b = uniform(lo);
    while (uu < u_end && nseg <= kMaxSeg) {
      while (uniform(s_pref[b + 1]) <= uu) ++b;
      const int len = uniform(s_len[b]);
      const int nt = (len + kIt - 1) / kIt;
      const int P = nt + kSegCost;
      const int r = uu - uniform(s_pref[b]);
      const int kvh = r / P;
      const int q = r - kvh * P;
      if (q < kSegCost) {
        uu += kSegCost - q;
        continue;
      }
      const int j0 = q - kSegCost;
      const int j1 = min(nt, j0 + (u_end - uu));
      if (nseg < kMaxSeg && tid == 0) s_desc[nseg] = SegDesc{b, kvh, len, j0, j1, nids};
      nids += (j1 * kIt - 1) / BS - j0 * kIt / BS + 1;
      ++nseg;
      uu += j1 - j0;
    }
  }
  if (nseg <= kMaxSeg && nids <= kRangeIds) {
    __syncthreads();
    for (int e = tid; e < nids; e += kThreads) {
      int sg = 0;
      while (sg + 1 < nseg && s_desc[sg + 1].id0 <= e) ++sg;
      const int b = s_desc[sg].b;
      const int j = s_desc[sg].j0 * kIt / BS + (e - s_desc[sg].id0);
      int id = -1;
      if (j * BS < s_desc[sg].len) {
        id = a.table[int64_t(b) * a.max_blocks + j];
        if (id < 0 || id >= a.n_local) {
          atomicAdd(a.err_count, 1);
          id = -1;
        }
      }
      s_rids[e] = id;
    }
    for (int e = tid; e < nseg * G * (kD / 8); e += kThreads) {   // 16-byte pieces of Q rows
      const int s2 = e / (G * (kD / 8));
      const int g = (e / (kD / 8)) % G;
      const int c = e % (kD / 8);
      const char* src = reinterpret_cast<const char*>(a.q) +
                        ((int64_t(s_desc[s2].b) * a.q_heads + s_desc[s2].kvh * G + g) * kD + c * 8) * 2;
      *reinterpret_cast<u32x4*>(&s_q[s2][g][c * 8]) = ld16(src);
    }
    __syncthreads();
    if (tid == 0) {
      for (int s2 = 0; s2 < nseg; ++s2) {
        const SegDesc& d = s_desc[s2];
        if (d.j0 != 0) continue;
        const int nt = (d.len + kIt - 1) / kIt;
        int32_t* info = a.info + (int64_t(d.b) * H + d.kvh) * 3;
        info[0] = int(blockIdx.x);
        info[1] = (s_pref[d.b] + d.kvh * (nt + kSegCost) + nt + kSegCost - 1) / per;
        info[2] = s2 == 0 ? 0 : 1;
      }
    }
    attend_range<G, BS, BF16>(a, s_desc, nseg, s_rids, s_q, sm,
                              [&](int s2, int g, int d, float M, float L, float O) {
      const SegDesc& sdd = s_desc[s2];
      const int nt = (sdd.len + kIt - 1) / kIt;
      if (sdd.j0 == 0 && sdd.j1 == nt) {
        store_out(a, (int64_t(sdd.b) * a.q_heads + sdd.kvh * G + g) * kD + d, L > 0.0f ? O / L : 0.0f);
      } else {
        const int64_t slot = int64_t(blockIdx.x) * 2 + (s2 == 0 ? 0 : 1);
        a.part_o[(slot * G + g) * kD + d] = O;
        if (d == 0) {
          a.part_ml[(slot * G + g) * 2] = M;
          a.part_ml[(slot * G + g) * 2 + 1] = L;
        }
      }
    });
    return;
  }

  int seg = 0;
  while (u < u_end) {
    int lo = 0, hi = B - 1;   // last sequence whose first unit is <= u
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_pref[mid] <= u) lo = mid;
      else hi = mid - 1;
    }
    const int b = uniform(lo);
    const int len = uniform(s_len[b]);
    const int nt = (len + kIt - 1) / kIt;
    const int P = nt + kSegCost;            // a pair's units: kSegCost, then its tiles
    const int r = u - uniform(s_pref[b]);
    const int kvh = r / P;
    const int q = r - kvh * P;
    if (q < kSegCost) {                      // cost units carry no tiles
      u += kSegCost - q;
      continue;
    }
    const int j0 = q - kSegCost;
    const int j1 = min(nt, j0 + (u_end - u));
    const bool whole = j0 == 0 && j1 == nt;
    const int64_t slot = int64_t(blockIdx.x) * 2 + (seg == 0 ? 0 : 1);
    attend_segment<G, BS, BF16>(a, b, kvh, len, j0, j1, sm,
                                [&](int g, int d, float M, float L, float O) {
      if (whole) {
        store_out(a, (int64_t(b) * a.q_heads + kvh * G + g) * kD + d, L > 0.0f ? O / L : 0.0f);
      } else {
        a.part_o[(slot * G + g) * kD + d] = O;
        if (d == 0) {
          a.part_ml[(slot * G + g) * 2] = M;
          a.part_ml[(slot * G + g) * 2 + 1] = L;
        }
      }
    });
    if (j0 == 0 && tid == 0) {
      int32_t* info = a.info + (int64_t(b) * H + kvh) * 3;
      info[0] = int(blockIdx.x);
      info[1] = (uniform(s_pref[b]) + kvh * P + P - 1) / per;
      info[2] = seg == 0 ? 0 : 1;
    }
    u += j1 - j0;
    ++seg;
  }
}

// Grid form for batches too large for the LDS work list: grid (chunk of
// kGridChunkTiles tiles, KV head, sequence); partials go to row
// (sequence, query head, chunk) and the split-K combine merges them.
template <int G, int BS, bool BF16>
__global__ __launch_bounds__(kThreads, 2) void attn_mfma_grid(AttnArgs a) {
  __shared__ Smem<G> sm;
  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int raw = a.seq_lens[b];
  const int len = clamp_len(raw, a);
  if (split == 0 && kvh == 0 && threadIdx.x == 0 && len != raw && raw > 0)
    atomicAdd(a.err_count, 1);
  if (len == 0) {
    if (split == 0 && kvh == 0) write_zeros(a, b);
    return;
  }
  const int nt = (len + kIt - 1) / kIt;
  const int j0 = split * kGridChunkTiles;
  if (j0 >= nt) return;
  const int j1 = min(nt, j0 + kGridChunkTiles);
  attend_segment<G, BS, BF16>(a, b, kvh, len, j0, j1, sm,
                              [&](int g, int d, float M, float L, float O) {
    const int hq = kvh * G + g;
    if (j0 == 0 && j1 == nt) {
      store_out(a, (int64_t(b) * a.q_heads + hq) * kD + d, L > 0.0f ? O / L : 0.0f);
    } else {
      const int64_t row = (int64_t(b) * a.q_heads + hq) * a.n_split + split;
      a.part_o[row * kD + d] = O;
      if (d == 0) {
        a.part_ml[row * 2] = M;
        a.part_ml[row * 2 + 1] = L;
      }
    }
  });
}

// Online merge of partials [0, n) of one output; K loads of each kind per
// memory round trip, branch-free (indices past n repeat the last partial and
// are given weight 0), so all K loads are in flight together.
template <int K>
__device__ __forceinline__ void merge_partials(const AttnArgs& a, int G, int g, int d, int wa,
                                               int sa, int n, float& M, float& L, float& O) {
  for (int j0 = 0; j0 < n; j0 += K) {
    float mm[K], ll[K], oo[K];
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const int i = min(j0 + j, n - 1);
      const int64_t slot = int64_t(wa + i) * 2 + (i == 0 ? sa : 0);
      mm[j] = a.part_ml[(slot * G + g) * 2];
      ll[j] = a.part_ml[(slot * G + g) * 2 + 1];
      oo[j] = a.part_o[(slot * G + g) * kD + d];
    }
#pragma unroll
    for (int j = 0; j < K; ++j)
      if (j0 + j >= n) mm[j] = -INFINITY;
    float Mb = M;
#pragma unroll
    for (int j = 0; j < K; ++j) Mb = fmaxf(Mb, mm[j]);
    if (Mb == -INFINITY) continue;
    const float f_old = M == -INFINITY ? 0.0f : exp2f(M - Mb);
    L *= f_old;
    O *= f_old;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const float f = mm[j] == -INFINITY ? 0.0f : exp2f(mm[j] - Mb);
      L = fmaf(f, ll[j], L);
      O = fmaf(f, oo[j], O);
    }
    M = Mb;
  }
}

// Merges the partials of every (sequence, KV head) the stream-K ranges cut.
// Grid (pair, output group): each thread owns one (head, channel) output.
// info says which workgroups hold the pair's partials (first == last: the
// pair was written whole, or the sequence is empty).
__global__ __launch_bounds__(kThreads) void attn_combine_streamk(AttnArgs a) {
  const int H = a.kv_heads;
  const int G = a.q_heads / H;
  const int pair = blockIdx.x;
  const int b = pair / H;
  const int kvh = pair - b * H;
  const int e = blockIdx.y * kThreads + threadIdx.x;
  const int32_t* info = a.info + int64_t(pair) * 3;
  const int wa = info[0], wb = info[1], sa = info[2];
  if (wb <= wa || e >= G * kD) return;
  const int g = e / kD;
  const int d = e % kD;
  const int n = wb - wa + 1;
  float M = -INFINITY, L = 0.0f, O = 0.0f;
  if (n <= 4)
    merge_partials<4>(a, G, g, d, wa, sa, n, M, L, O);
  else
    merge_partials<16>(a, G, g, d, wa, sa, n, M, L, O);
  store_out(a, (int64_t(b) * a.q_heads + kvh * G + g) * kD + d, L > 0.0f ? O / L : 0.0f);
}


template <int G, int BS, bool BF16>
hipError_t launch_typed(const AttnArgs& a, hipStream_t stream) {
  if (a.stream_k) {
    const int grid = attn_streamk_grid();
    hipLaunchKernelGGL((attn_mfma_streamk<G, BS, BF16>), dim3(grid), dim3(kThreads), 0, stream,
                       a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int groups = (a.q_heads / a.kv_heads * kD + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(attn_combine_streamk, dim3(a.batch * a.kv_heads, groups), dim3(kThreads),
                       0, stream, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((attn_mfma_grid<G, BS, BF16>), dim3(a.n_split, a.kv_heads, a.batch),
                     dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split <= 1) return e;
  return launch_attn_combine(a, stream);
}

template <int G, int BS>
hipError_t launch_g_bs(const AttnArgs& a, hipStream_t stream) {
  return a.dtype == 1 ? launch_typed<G, BS, true>(a, stream) : launch_typed<G, BS, false>(a, stream);
}

template <int G>
hipError_t launch_g(const AttnArgs& a, hipStream_t stream) {
  switch (a.block_size) {
    case 16: return launch_g_bs<G, 16>(a, stream);
    case 32: return launch_g_bs<G, 32>(a, stream);
    case 64: return launch_g_bs<G, 64>(a, stream);
    case 128: return launch_g_bs<G, 128>(a, stream);
    case 256: return launch_g_bs<G, 256>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// Stream-K grid: one workgroup per CU. A second resident workgroup per CU
// adds no bandwidth (the two share the CU's memory path, the second running
// about 20 % slower) but doubles the cut pairs and their partials.
int attn_streamk_grid() {
  static const int grid = [] {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      return 256;
    return std::min(cus, kMaxStreamGrid);
  }();
  return grid;
}

// The fixed workspace of the no-allocation entry point. Host code never uses
// this name as an address: it takes the per-device address from
// noalloc_workspace().
__device__ __align__(256) unsigned char scratch[kNoAllocBytes];

hipError_t noalloc_workspace(void** ptr) {
  static std::mutex mu;
  static std::unordered_map<int, void*> addr;   // device -> address of `scratch` there
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    it = addr.emplace(dev, p).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

hipError_t launch_paged_attention_mfma(const AttnArgs& a, hipStream_t stream) {
  if (a.batch == 0) return hipSuccess;
  switch (a.q_heads / a.kv_heads) {
    case 1: return launch_g<1>(a, stream);
    case 2: return launch_g<2>(a, stream);
    case 4: return launch_g<4>(a, stream);
    case 8: return launch_g<8>(a, stream);
    case 16: return launch_g<16>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ema
