// Launchers of the gfx950 kernels. All take device pointers and enqueue on
// `stream`; none allocates.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace ema {

// The two pools as the kernels see them.
struct PoolView {
  char* local;           // n_local blocks, EMA_LAYOUT_ATTN
  char* slice;           // n_slice blocks, slice_layout
  int64_t block_bytes;
  int32_t n_local;
  int32_t n_slice;
  int32_t kv_heads;
  int32_t block_size;
  int32_t slice_layout;  // 0 ATTN, 1 NHD
};

// Reclaim's table rewrite, done by the first `n_groups` workgroups of the
// reclaim's copy launch (so the rewrite costs no launch of its own): every
// entry t of tables[n_entries] with base <= t < base + n_range becomes
// range_map[t - base] (the mover's destination, -1 for a preempted sequence's
// block, else t); any other t >= 0 with bits_base <= t < bits_base + n_bits
// becomes -1 when bit t - bits_base of released_bits is set (a released block
// outside the range: one load per entry, whatever the number released).
// n_groups == 0: no rewrite.
struct TableRewrite {
  int32_t* tables = nullptr;
  int64_t n_entries = 0;
  const int32_t* range_map = nullptr;
  const uint32_t* released_bits = nullptr;
  int32_t base = 0;
  int32_t n_range = 0;            // range_map == nullptr: the range maps through the
                                  // launch's copy runs (t in run r -> run_dst[r] + offset)
  int32_t bits_base = 0;
  int32_t n_bits = 0;
  int32_t n_groups = 0;
};
constexpr int kRewriteEntries = 8192;   // table entries per rewriting workgroup

// Where copy i's source and destination come from: device id lists, or a few
// contiguous runs carried in the launch's own arguments, so that a plan of
// long runs (a reclaim of a contiguous range, a slab swap) needs no upload.
constexpr int kArgRuns = 24;
struct CopyIds {
  const int32_t* src = nullptr;   // device [n] (n_runs == 0)
  const int32_t* dst = nullptr;   // device [n]; nullptr: dst_base + i (n_runs == 0)
  int32_t dst_base = 0;
  int32_t n_runs = 0;             // > 0: copy i lies in run r, run_off[r] <= i < run_off[r + 1]
  int32_t run_src[kArgRuns] = {};
  int32_t run_dst[kArgRuns] = {};
  int32_t run_off[kArgRuns + 1] = {};
};

// dst[i] <- src[i] for i < n (unified ids), re-laid between pool layouts.
// Ids outside [0, n_local + n_slice) are skipped and counted in *err_count.
// `runs`: the lists are mostly ascending runs of ids (reclaim moves,
// contiguous-run prefetches) rather than scattered blocks; only the work
// distribution depends on it. `rw` (optional): the table rewrite to run in the
// same launch (n_groups is set by the launcher). dst == nullptr: the
// destinations are dst_base + i (a contiguous staging image).
hipError_t launch_block_copy(const PoolView& pv, const int32_t* src, const int32_t* dst,
                             int32_t n, int32_t* err_count, hipStream_t stream,
                             bool runs = false, const TableRewrite* rw = nullptr,
                             int32_t dst_base = 0);
// The same for n copies given as contiguous runs (src_first[r], dst_first[r],
// len[r]), r < n_runs <= kArgRuns, carried in the launch arguments.
hipError_t launch_block_copy_runs(const PoolView& pv, const int32_t* src_first,
                                  const int32_t* dst_first, const int32_t* len, int32_t n_runs,
                                  int32_t* err_count, hipStream_t stream,
                                  const TableRewrite* rw = nullptr);

// New decode token of every sequence into its block (ATTN layout): row
// (len-1) % bs of local block table[b][(len-1) / bs], len = seq_lens[b] > 0.
// Out-of-range block indices or ids are skipped and counted in *err_count.
hipError_t launch_kv_append(const PoolView& pv, const void* k_new, const void* v_new,
                            const int32_t* table, const int32_t* seq_lens, int32_t batch,
                            int32_t max_blocks, int32_t* err_count, hipStream_t stream);

struct AttnArgs {
  const void* q;            // [B][Hq][128] 16-bit
  const int32_t* table;     // [B][max_blocks]
  const int32_t* seq_lens;  // [B]
  void* out;                // [B][Hq][128], out_dtype
  float* part_o;            // [B][Hq][n_split][128] split-K partial outputs
  float* part_ml;           // [B][Hq][n_split][2] running max (log2 domain) and sum
                            // (stream-K: [2 * grid][G][...] partial slots instead)
  int32_t* info;            // stream-K: [B][Hkv][3] first / last workgroup, first slot
  int32_t* err_count;
  const char* local;        // local pool base
  int64_t block_bytes;
  int32_t n_local;
  int32_t batch, q_heads, kv_heads, block_size, max_blocks, n_split, dtype;
  int32_t chunk;            // tokens per split (grid forms)
  int32_t stream_k;         // matrix-core kernel: stream-K scheduling (else grid form)
  int32_t out_dtype;        // kOutF32, kOutF16 or kOutBF16
  float scale_log2;         // softmax scale times log2(e)
};

// Output element types (the values of EMA_F16, EMA_BF16, EMA_F32).
constexpr int kOutF16 = 0;
constexpr int kOutBF16 = 1;
constexpr int kOutF32 = 2;

constexpr int kMfmaGridChunk = 1024;   // tokens per workgroup of the matrix-core grid form
// Sequences the stream-K work list holds in LDS (lengths and prefix sums):
// sized so that a workgroup's LDS stays within half a CU's 160 KiB, which
// every call measured faster (16 query heads per KV head need twice the
// merge space, hence the smaller list).
constexpr int streamk_max_batch(int group) { return group >= 16 ? 2048 : 4096; }
constexpr int kMaxStreamGrid = 2048;   // stream-K workgroups (partial slots: 2 each)
constexpr int kHeadDim = 128;          // the only head size the device paths take
constexpr int kMaxGroup = 16;          // query heads per KV head
// Stream-K workgroups of every call in this process: one per CU of the device
// current at the first call, at most kMaxStreamGrid. Partial slots: 2 per
// workgroup, each kMaxGroup x (kHeadDim + 2) floats at most.
int attn_streamk_grid();

// Fixed attention workspace for callers that cannot allocate: a file-scope
// device array (one per GPU, held until the process ends) with partial slots
// for up to kNoAllocGrid stream-K workgroups at kMaxGroup query heads per KV
// head, followed by combine records for kNoAllocPairs (sequence, KV head)
// pairs. Every call writes each record it reads, so nothing in it needs
// clearing; calls that overlap on one GPU race on it.
constexpr int kNoAllocGrid = 512;
constexpr int kNoAllocPairs = 32768;
constexpr size_t kNoAllocPartFloats = size_t(2) * kNoAllocGrid * kMaxGroup * (kHeadDim + 2);
constexpr size_t kNoAllocBytes = kNoAllocPartFloats * 4 + size_t(kNoAllocPairs) * 3 * 4;
// Device address of that array on the current device (looked up once per
// device with hipGetSymbolAddress, then cached).
hipError_t noalloc_workspace(void** ptr);

// Matrix-core kernel: stream-K when stream_k is set, else the grid form with
// chunk == kMfmaGridChunk.
hipError_t launch_paged_attention_mfma(const AttnArgs& a, hipStream_t stream);
// Merges the split-K partials of sequences longer than one chunk.
hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t stream);

}  // namespace ema
