// Block-table-driven gather/scatter of layer-blocks between the local pool and
// the slice (prefetch before use, migration, reclaim write-back / compaction).
//
// When both pools share one layout (the slice in the local layout), every
// copy is a straight 16-byte-per-lane copy: a wavefront moves 2 KiB of a
// block (two wave instructions of 1 KiB each way, fully coalesced; 1, 4, 8
// and 16 KiB per wavefront move fewer bytes per second). Lists of up to 2^22
// pieces (8 GiB) of scattered blocks of up to 64 KiB go one wavefront per
// workgroup, which spreads each block over all XCDs; long ascending runs,
// larger blocks and larger lists go four wavefronts (8 KiB contiguous) per
// workgroup, which measured faster or steadier for them.
//
// Otherwise the work unit is 4 KiB of one destination block, i.e. 16 tokens x
// 128 channels of one KV head's K or V -- one block-row at block size 16. One
// wavefront owns a unit, four per workgroup. Same-layout units are straight
// copies as above. Units that change layout go through the wave's LDS tile:
// K rows only change order (256-byte rows are re-addressed, no LDS), V is
// transposed between [token][channel] (NHD) and [channel][token] (ATTN) in
// LDS so that both the global reads and the global writes stay 16 bytes per
// lane. Into ATTN, a V unit is T = min(BS, 64) tokens of 2048/T channels: its
// transposed rows are written whole up to 64 tokens (128 B), its token rows
// are read 64 B or more at a time, and the four units of a workgroup cover
// whole 256-B token rows; out of ATTN it is 16 tokens of all 128 channels
// (whole token rows written), or from block size 64 on 32 tokens of 64
// channels (128-B pieces of token rows written). The tile is dynamic LDS, requested only
// when the slice layout differs from the local one.
#include "kernels.h"

#include <algorithm>

namespace ema {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kUnitBytes = 4096;    // work unit of the layout-changing kernel
constexpr int kPieceBytes = 2048;   // work unit of the same-layout kernel
constexpr int kWaves = 4;
constexpr int kTileRow = 128 + 8;   // u16 per LDS tile row (padded, keeps 16 B alignment)

// Tokens of one V unit into the local layout: whole transposed rows up to 64
// tokens (128 B); with larger blocks a unit is 64 tokens x 32 channels, and
// the four units of a workgroup cover one token group's 128 channels.
__host__ __device__ constexpr int v_unit_tokens(int bs) { return bs < 64 ? bs : 64; }

// u16 per wave of the relayout tile: 16 x kTileRow or 32 x 72 (out of ATTN),
// T x (2048/T + 8), T = v_unit_tokens(bs) (into ATTN).
__host__ __device__ constexpr int tile_elems(int bs) {
  return 16 * kTileRow > 2048 + 8 * v_unit_tokens(bs) ? 16 * kTileRow
                                                      : 2048 + 8 * v_unit_tokens(bs);
}

// Block data is touched once per copy: streaming (non-temporal) loads and
// stores keep it from displacing other data in L2 and the memory-side cache,
// and keep written lines from being flushed later under another kernel's reads.
__device__ __forceinline__ u32x4 ld16(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st16(char* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// LDS writes of this wave must land before other lanes of the wave read them.
__device__ __forceinline__ void wave_lds_sync() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Source and destination of copy i (wave-uniform i).
__device__ __forceinline__ void copy_ids(const CopyIds& c, int32_t i, int32_t& s, int32_t& d) {
  if (c.n_runs > 0) {
    int r = 0;
    for (int q = 1; q < c.n_runs; ++q)
      if (c.run_off[q] <= i) r = q;
    s = c.run_src[r] + (i - c.run_off[r]);
    d = c.run_dst[r] + (i - c.run_off[r]);
  } else {
    s = c.src[i];
    d = c.dst ? c.dst[i] : c.dst_base + i;
  }
}

// The table-rewrite share of a reclaim launch: workgroup g rewrites entries
// [g * kRewriteEntries, (g + 1) * kRewriteEntries), threads strided so that
// reads and writes stay coalesced. Only changed entries are written.
__device__ __forceinline__ void rewrite_tables(const TableRewrite& rw, const CopyIds& ids, int g) {
  const int64_t e0 = int64_t(g) * kRewriteEntries;
  const int64_t e1 = e0 + kRewriteEntries < rw.n_entries ? e0 + kRewriteEntries : rw.n_entries;
  for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
    const int32_t t = rw.tables[e];
    if (t < 0) continue;
    int32_t nt = t;
    const uint32_t r = uint32_t(t - rw.base);
    if (r < uint32_t(rw.n_range)) {
      if (rw.range_map) {
        nt = rw.range_map[r];
      } else {                                   // movers: the launch's copy runs
        for (int q = 0; q < ids.n_runs; ++q) {
          const int32_t o = t - ids.run_src[q];
          const int32_t len = ids.run_off[q + 1] - ids.run_off[q];
          if (o >= 0 && o < len) nt = ids.run_dst[q] + o;
        }
      }
    } else if (uint32_t(t - rw.bits_base) < uint32_t(rw.n_bits)) {
      const uint32_t b = uint32_t(t - rw.bits_base);
      if ((rw.released_bits[b >> 5] >> (b & 31)) & 1u) nt = -1;
    }
    if (nt != t) rw.tables[e] = nt;
  }
}

__global__ __launch_bounds__(256) void block_copy_kernel(PoolView pv, CopyIds ids,
                                                         int32_t n, int32_t* err_count,
                                                         TableRewrite rw) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds_tile[];
  if (int(blockIdx.x) < rw.n_groups) {
    rewrite_tables(rw, ids, blockIdx.x);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int upb = int(pv.block_bytes / kUnitBytes);
  const int64_t unit = (int64_t(blockIdx.x) - rw.n_groups) * kWaves + wave;
  if (unit >= int64_t(n) * upb) return;
  const int32_t i = int32_t(unit / upb);
  const int k = int(unit - int64_t(i) * upb);
  int32_t s, d;
  copy_ids(ids, __builtin_amdgcn_readfirstlane(i), s, d);
  const int32_t n_total = pv.n_local + pv.n_slice;
  if (s < 0 || s >= n_total || d < 0 || d >= n_total) {
    if (k == 0 && lane == 0) atomicAdd(err_count, 1);
    return;
  }
  const bool s_local = s < pv.n_local;
  const bool d_local = d < pv.n_local;
  const char* sb = s_local ? pv.local + int64_t(s) * pv.block_bytes
                           : pv.slice + int64_t(s - pv.n_local) * pv.block_bytes;
  char* db = d_local ? pv.local + int64_t(d) * pv.block_bytes
                     : pv.slice + int64_t(d - pv.n_local) * pv.block_bytes;
  const int s_nhd = s_local ? 0 : pv.slice_layout;
  const int d_nhd = d_local ? 0 : pv.slice_layout;

  if (s_nhd == d_nhd) {
    const int64_t off = int64_t(k) * kUnitBytes + lane * 16;
    const u32x4 v0 = ld16(sb + off);
    const u32x4 v1 = ld16(sb + off + 1024);
    const u32x4 v2 = ld16(sb + off + 2048);
    const u32x4 v3 = ld16(sb + off + 3072);
    st16(db + off, v0);
    st16(db + off + 1024, v1);
    st16(db + off + 2048, v2);
    st16(db + off + 3072, v3);
    return;
  }

  // Layout change. Unit k -> (half, head h, group tg): a 16-token group, or
  // for V into ATTN a group of T tokens x 2048/T channels (BS/16 groups
  // either way).
  const int H = pv.kv_heads;
  const int BS = pv.block_size;
  const int tgs = BS / 16;
  const int uph = H * tgs;
  const int half = k / uph;
  const int r = k - half * uph;
  const int h = r / tgs;
  const int tg = r - h * tgs;
  const int64_t half_bytes = pv.block_bytes / 2;

  if (half == 0) {
    // K: 16 rows of 256 B; ATTN row (h, t) at (h*BS + t)*256, NHD row at (t*H + h)*256.
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = tg * 16 + j * 4 + (lane >> 4);
      const int64_t row = s_nhd ? int64_t(t * H + h) : int64_t(h * BS + t);
      v[j] = ld16(sb + row * 256 + (lane & 15) * 16);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = tg * 16 + j * 4 + (lane >> 4);
      const int64_t row = d_nhd ? int64_t(t * H + h) : int64_t(h * BS + t);
      st16(db + row * 256 + (lane & 15) * 16, v[j]);
    }
    return;
  }

  uint16_t* tw = lds_tile + wave * tile_elems(BS);
  const char* sv = sb + half_bytes;
  char* dv = db + half_bytes;
  if (s_nhd) {
    // NHD -> ATTN, unit (h, token group, channel group): T = v_unit_tokens(BS)
    // tokens of C = 2048/T channels. Read C channels of each of the T token
    // rows (LR lanes per row) into the tile as [t][c], then write C
    // transposed rows of T tokens (LC lanes each): reads and writes stay at
    // least 64 B contiguous, and the four waves of a workgroup read whole
    // 256-B token rows between them.
    const int T = v_unit_tokens(BS);
    const int C = 2048 / T;
    const int cgs = 128 / C;                  // channel groups per token group
    const int t_base = (tg / cgs) * T;
    const int c0 = (tg % cgs) * C;
    const int LR = C / 8;
    const int stride = C + 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = j * (64 / LR) + lane / LR;
      const int c = (lane % LR) * 8;
      const u32x4 v = ld16(sv + (int64_t((t_base + t) * H + h) * 128 + c0 + c) * 2);
      *reinterpret_cast<u32x4*>(&tw[t * stride + c]) = v;
    }
    wave_lds_sync();
    const int LC = T / 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int item = j * 64 + lane;
      const int cc = item / LC;
      const int t0 = (item % LC) * 8;
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = uint32_t(tw[(t0 + 2 * q) * stride + cc]) |
               (uint32_t(tw[(t0 + 2 * q + 1) * stride + cc]) << 16);
      const u32x4 out = {w[0], w[1], w[2], w[3]};
      st16(dv + (int64_t(h * 128 + c0 + cc) * BS + t_base + t0) * 2, out);
    }
  } else {
    // ATTN -> NHD, unit (h, token group, channel group): T = 16 tokens of all
    // 128 channels, or from block size 64 on T = 32 tokens of 64 channels.
    // Read the unit's C channel rows of T tokens (T/8 lanes per row), scatter
    // into the tile as [t][c], then write T token rows of C channels (C/8
    // lanes per row): whole 256-B token rows at T = 16; at T = 32, 64-B
    // channel-row reads and 128-B token-row writes (measured faster than
    // 64 tokens of 32 channels, whose writes are 64 B).
    const int T = BS >= 64 ? 32 : 16;
    const int C = 2048 / T;
    const int cgs = 128 / C;
    const int t_base = (tg / cgs) * T;
    const int c0 = (tg % cgs) * C;
    const int IR = T / 8;                     // 16-B items per channel row
    const int stride = C + 8;
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int item = j * 64 + lane;
      const int c = item / IR;
      const int t0 = (item % IR) * 8;
      v[j] = ld16(sv + (int64_t(h * 128 + c0 + c) * BS + t_base + t0) * 2);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int item = j * 64 + lane;
      const int c = item / IR;
      const int t0 = (item % IR) * 8;
      const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        tw[(t0 + 2 * q) * stride + c] = uint16_t(w[q] & 0xffffu);
        tw[(t0 + 2 * q + 1) * stride + c] = uint16_t(w[q] >> 16);
      }
    }
    wave_lds_sync();
    const int LW = C / 8;                     // lanes per token row written
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tl = j * (64 / LW) + lane / LW;
      const int cp = (lane % LW) * 8;
      const u32x4 out = *reinterpret_cast<const u32x4*>(&tw[tl * stride + cp]);
      st16(dv + (int64_t((t_base + tl) * H + h) * 128 + c0 + cp) * 2, out);
    }
  }
}

// Same-layout copy (both pools in the local layout): wave w of workgroup g
// (blockDim.x / 64 waves each) moves piece g * (blockDim.x / 64) + w, 2 KiB of
// block src_ids[i] to the same offset of block dst_ids[i]. Out-of-range ids
// are skipped and counted once per block.
__global__ __launch_bounds__(256) void block_copy_same_kernel(PoolView pv, CopyIds ids,
                                                              int32_t n, int32_t* err_count,
                                                              TableRewrite rw) {
  if (int(blockIdx.x) < rw.n_groups) {
    rewrite_tables(rw, ids, blockIdx.x);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int ppb = int(pv.block_bytes / kPieceBytes);
  const int64_t piece =
      (int64_t(blockIdx.x) - rw.n_groups) * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (piece >= int64_t(n) * ppb) return;
  const int32_t i = int32_t(piece / ppb);
  const int k = int(piece - int64_t(i) * ppb);
  int32_t s, d;
  copy_ids(ids, __builtin_amdgcn_readfirstlane(i), s, d);
  const int32_t n_total = pv.n_local + pv.n_slice;
  if (s < 0 || s >= n_total || d < 0 || d >= n_total) {
    if (k == 0 && lane == 0) atomicAdd(err_count, 1);
    return;
  }
  const char* sb = s < pv.n_local ? pv.local + int64_t(s) * pv.block_bytes
                                  : pv.slice + int64_t(s - pv.n_local) * pv.block_bytes;
  char* db = d < pv.n_local ? pv.local + int64_t(d) * pv.block_bytes
                            : pv.slice + int64_t(d - pv.n_local) * pv.block_bytes;
  const int64_t off = int64_t(k) * kPieceBytes + lane * 16;
  const u32x4 v0 = ld16(sb + off);
  const u32x4 v1 = ld16(sb + off + 1024);
  st16(db + off, v0);
  st16(db + off + 1024, v1);
}

// One workgroup per (sequence, KV head), one thread per channel: the K element
// goes to the token's row, the V element to the token's column of the
// transposed V rows.
__global__ __launch_bounds__(128) void kv_append_kernel(PoolView pv, const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new,
                                                        const int32_t* __restrict__ table,
                                                        const int32_t* __restrict__ seq_lens,
                                                        int32_t max_blocks, int32_t* err_count) {
  const int b = blockIdx.x;
  const int h = blockIdx.y;
  const int d = threadIdx.x;
  const int H = pv.kv_heads;
  const int BS = pv.block_size;
  const int len = seq_lens[b];
  if (len <= 0) return;
  const int p = len - 1;
  const int j = p / BS;
  const int32_t id = j < max_blocks ? table[int64_t(b) * max_blocks + j] : -1;
  if (id < 0 || id >= pv.n_local) {
    if (h == 0 && d == 0) atomicAdd(err_count, 1);
    return;
  }
  const int r = p - j * BS;
  uint16_t* blk = reinterpret_cast<uint16_t*>(pv.local + int64_t(id) * pv.block_bytes);
  const int64_t src = (int64_t(b) * H + h) * 128 + d;
  blk[(int64_t(h) * BS + r) * 128 + d] = k_new[src];
  blk[int64_t(BS) * H * 128 + (int64_t(h) * 128 + d) * BS + r] = v_new[src];
}

}  // namespace

namespace {

hipError_t launch_copy(const PoolView& pv, CopyIds ids, int32_t n, int32_t* err_count,
                       hipStream_t stream, bool runs, const TableRewrite* rw) {
  TableRewrite rwl;
  if (rw && rw->n_entries > 0) {
    rwl = *rw;
    rwl.n_groups = int32_t((rw->n_entries + kRewriteEntries - 1) / kRewriteEntries);
  }
  if (n <= 0 && rwl.n_groups == 0) return hipSuccess;
  const bool same = pv.slice_layout == 0;
  const int64_t upb = pv.block_bytes / (same ? kPieceBytes : kUnitBytes);   // waves per block
  const int wg_waves =
      same && !runs && pv.block_bytes <= 65536 && int64_t(n) * upb <= (int64_t(1) << 22) ? 1
                                                                                        : kWaves;
  const size_t lds = same ? 0 : size_t(kWaves) * tile_elems(pv.block_size) * 2;
  // A launch stays below 2^32 work-items: at most 2^25 wavefronts. The table
  // rewrite rides on the first launch; lists are split, run plans always fit.
  const int64_t max_blocks = std::max<int64_t>(1, (int64_t(1) << 25) / upb);
  if (ids.n_runs > 0 && n > max_blocks) return hipErrorInvalidValue;
  int64_t b0 = 0;
  do {
    const int32_t m = int32_t(std::max<int64_t>(0, std::min<int64_t>(max_blocks, n - b0)));
    const int64_t grid = (int64_t(m) * upb + wg_waves - 1) / wg_waves + rwl.n_groups;
    const unsigned threads = same ? unsigned(64 * wg_waves) : 256u;
    CopyIds part = ids;
    if (ids.n_runs == 0) {
      part.src = m ? ids.src + b0 : nullptr;
      part.dst = m && ids.dst ? ids.dst + b0 : nullptr;
      part.dst_base = ids.dst ? 0 : int32_t(ids.dst_base + b0);
    }
    if (same)
      hipLaunchKernelGGL(block_copy_same_kernel, dim3(unsigned(grid)), dim3(threads), 0, stream,
                         pv, part, m, err_count, rwl);
    else
      hipLaunchKernelGGL(block_copy_kernel, dim3(unsigned(grid)), dim3(threads), lds, stream, pv,
                         part, m, err_count, rwl);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    rwl.n_groups = 0;
    b0 += m;
  } while (b0 < n);
  return hipSuccess;
}

}  // namespace

hipError_t launch_block_copy(const PoolView& pv, const int32_t* src, const int32_t* dst,
                             int32_t n, int32_t* err_count, hipStream_t stream, bool runs,
                             const TableRewrite* rw, int32_t dst_base) {
  CopyIds ids;
  ids.src = src;
  ids.dst = dst;
  ids.dst_base = dst_base;
  return launch_copy(pv, ids, n, err_count, stream, runs, rw);
}

hipError_t launch_block_copy_runs(const PoolView& pv, const int32_t* src_first,
                                  const int32_t* dst_first, const int32_t* len, int32_t n_runs,
                                  int32_t* err_count, hipStream_t stream,
                                  const TableRewrite* rw) {
  if (n_runs < 0 || n_runs > kArgRuns) return hipErrorInvalidValue;
  CopyIds ids;
  ids.n_runs = n_runs;
  int64_t n = 0;
  for (int32_t r = 0; r < n_runs; ++r) {
    ids.run_src[r] = src_first[r];
    ids.run_dst[r] = dst_first[r];
    ids.run_off[r] = int32_t(n);
    n += len[r];
  }
  ids.run_off[n_runs] = int32_t(n);
  if (n > INT32_MAX) return hipErrorInvalidValue;
  return launch_copy(pv, ids, int32_t(n), err_count, stream, true, rw);
}

hipError_t launch_kv_append(const PoolView& pv, const void* k_new, const void* v_new,
                            const int32_t* table, const int32_t* seq_lens, int32_t batch,
                            int32_t max_blocks, int32_t* err_count, hipStream_t stream) {
  if (batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_append_kernel, dim3(unsigned(batch), unsigned(pv.kv_heads)), dim3(128), 0,
                     stream, pv, static_cast<const uint16_t*>(k_new),
                     static_cast<const uint16_t*>(v_new), table, seq_lens, max_blocks, err_count);
  return hipGetLastError();
}

}  // namespace ema
