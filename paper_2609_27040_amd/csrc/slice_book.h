// Host bookkeeping of one memory slice plus the local paged cache: owner tags,
// lowest-free allocation, lending, validation of copy lists and the reclaim
// planner. Pure C++ (no HIP): the device side only executes the copy lists and
// table remaps this produces.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace ema {

constexpr int32_t kFree = -1;
constexpr int32_t kStaging = -2;
constexpr int32_t kLender = -3;

constexpr int kOk = 0;
constexpr int kErrInval = -1;
constexpr int kErrNomem = -2;
constexpr int kErrOwner = -3;
constexpr int kErrHip = -4;

// Free-slot set over [0, n) with "n lowest members" queries: one bit per slot.
class FreeBits {
 public:
  void reset(int32_t n, bool all_free);
  void set(int32_t i, bool is_free);
  bool get(int32_t i) const { return (w_[i >> 6] >> (i & 63)) & 1ull; }
  int32_t count() const { return count_; }
  // Lowest `k` free slots below `limit`, ascending; returns how many were found.
  int32_t lowest(int32_t k, int32_t limit, int32_t* out) const;
  int32_t count_below(int32_t limit) const;

 private:
  std::vector<uint64_t> w_;
  int32_t n_ = 0;
  int32_t count_ = 0;
};

constexpr int32_t kBorrowed = -4;   // slab tag: the borrower's

// Slab management of the slice (slab_book.cpp). A slab is S positions, the
// same positions in every one of L layers; group = layers per layer group.
struct SlabCfg {
  int32_t layers = 0, slab_blocks = 0, group = 0, layout = 0;   // 0 layer-, 1 slab-, 2 group-major
};

struct SlabReclaimPlan {
  int32_t reclaimed = 0;
  std::vector<int32_t> slabs;          // slabs taken by the lender, in order
  std::vector<int32_t> victims;        // preempted owners, in order
  std::vector<int32_t> released;       // every block they held, unified ids, ascending
};

struct ReclaimPlan {
  int32_t reclaimed = 0;
  int32_t cut = 0;
  int32_t written_back = 0;
  std::vector<int32_t> move_src;      // unified ids, ascending
  std::vector<int32_t> move_dst;      // unified ids
  std::vector<int32_t> victims;       // preempted owners, in order
  std::vector<int32_t> victim_blocks; // every block they held, unified ids
};

class SliceBook {
 public:
  void init(int32_t n_local, int32_t n_slice);

  int32_t n_local() const { return n_local_; }
  int32_t n_slice() const { return n_slice_; }
  int32_t lim() const { return lim_; }
  int32_t free_local() const { return free_local_.count(); }
  int32_t free_slice() const { return free_slice_.count(); }
  int32_t owner(int32_t u) const { return u < n_local_ ? own_local_[u] : own_slice_[u - n_local_]; }
  bool in_range(int64_t u) const { return u >= 0 && u < int64_t(n_local_) + n_slice_; }
  const std::vector<int32_t>& own_local() const { return own_local_; }
  const std::vector<int32_t>& own_slice() const { return own_slice_; }

  int alloc(int32_t pool, int32_t n, const int32_t* owners, int32_t* out_ids, std::string* err);
  int free_blocks(const int32_t* ids, int32_t n, std::string* err);
  int lend(int32_t n, int32_t* added, std::string* err);
  // Copy-list checks (pure reads of state).
  int check_prefetch(const int32_t* src, const int32_t* dst, int32_t n, std::string* err) const;
  int check_migrate(const int32_t* src, const int32_t* dst, int32_t n, std::string* err) const;
  int check_writeback(const int32_t* src, const int32_t* dst, int32_t n, std::string* err) const;
  // Plans reclaim(n) and commits it to the owner tags.
  int reclaim(int32_t n, ReclaimPlan* plan, std::string* err);

  // ---- slab mode (slab_book.cpp) ----
  bool slab_mode() const { return slab_mode_; }
  const SlabCfg& slab_cfg() const { return cfg_; }
  int32_t n_slabs() const { return n_slabs_; }
  int64_t slab_version() const { return slab_version_; }
  const std::vector<int32_t>& slab_tag() const { return slab_tag_; }
  const std::vector<int32_t>& pos_owner() const { return pos_owner_; }
  // Switches an untouched slice (every slot FREE, lim = n_slice) to slabs.
  int slab_init(const SlabCfg& cfg, std::string* err);
  int slab_alloc(int32_t n, const int32_t* owners, int32_t* out_pos, std::string* err);
  int slab_free(const int32_t* pos, int32_t n, std::string* err);
  int slab_reclaim(int32_t n, SlabReclaimPlan* plan, std::string* err);
  // Slice slot of (slab i, layer l, position p).
  int64_t slab_slot(int32_t i, int32_t l, int32_t p) const;
  // Borrowed slabs in index order.
  std::vector<int32_t> borrowed_slabs() const;
  // Offset inside a group's staging image of (borrowed rank r of m, group layer j, position p).
  int64_t stage_index(int32_t r, int32_t m, int32_t j, int32_t p) const;
  // Source unified ids of group g's swap, in staging order (m * group * S of them).
  void group_sources(int32_t g, std::vector<int32_t>* src) const;

 private:
  void set_owner(int32_t u, int32_t o);
  int check_pairs(const int32_t* src, const int32_t* dst, int32_t n, std::string* err) const;

  void set_pos(int32_t pos, int32_t o);
  void set_slab(int32_t i, int32_t tag);
  void release_if_empty(int32_t i);

  int32_t n_local_ = 0, n_slice_ = 0, lim_ = 0;
  std::vector<int32_t> own_local_, own_slice_;
  FreeBits free_local_, free_slice_;   // slice bits only below lim_
  bool slab_mode_ = false;
  SlabCfg cfg_;
  int32_t n_slabs_ = 0;
  int64_t slab_version_ = 0;           // bumped whenever the set of borrowed slabs changes
  std::vector<int32_t> slab_tag_;      // kLender, kFree or kBorrowed
  std::vector<int32_t> pos_owner_;     // n_slabs * S: owner or kFree
  std::vector<int32_t> slab_used_;     // used positions per slab
};

}  // namespace ema
