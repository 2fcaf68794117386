// Slab management of the slice (section 4.2.1-4.2.3): see slice_book.h.
//
// A slab is S block positions, the same positions in every one of the cache's
// L layers, and belongs to one user at a time: the lender, nobody (lent but
// unused) or the borrower. A borrowed slab's positions each hold one logical
// block of one sequence (all L layers of it) or are free; a slab whose last
// position is freed returns to the slice. The per-slot owner tags of the slice
// are kept in step with the slab state, so the copy-list checks of the block
// mode apply to slab-resident blocks unchanged.
//
// Placement of (slab i, layer l, position p), n slabs, k layers per group:
//   layer-major        (l * n + i) * S + p
//   slab-major         (i * L + l) * S + p
//   layer-group-major  ((l / k * n + i) * k + l % k) * S + p
// The swap of layer group g fills a staging image of the m borrowed slabs in
// the layout's own order: (j * m + r) * S + p for layer-major, (r * k + j) * S
// + p otherwise (r: rank of the slab among the borrowed ones, j: layer in the
// group), so that contiguous slice ranges stay contiguous in staging.
#include <algorithm>

#include "slice_book.h"

namespace ema {

int64_t SliceBook::slab_slot(int32_t i, int32_t l, int32_t p) const {
  const int64_t n = n_slabs_, S = cfg_.slab_blocks, L = cfg_.layers, k = cfg_.group;
  switch (cfg_.layout) {
    case 0: return (int64_t(l) * n + i) * S + p;
    case 1: return (int64_t(i) * L + l) * S + p;
    default: return ((int64_t(l / k) * n + i) * k + l % k) * S + p;
  }
}

int64_t SliceBook::stage_index(int32_t r, int32_t m, int32_t j, int32_t p) const {
  const int64_t S = cfg_.slab_blocks;
  if (cfg_.layout == 0) return (int64_t(j) * m + r) * S + p;
  return (int64_t(r) * cfg_.group + j) * S + p;
}

std::vector<int32_t> SliceBook::borrowed_slabs() const {
  std::vector<int32_t> out;
  for (int32_t i = 0; i < n_slabs_; ++i)
    if (slab_tag_[i] == kBorrowed) out.push_back(i);
  return out;
}

void SliceBook::group_sources(int32_t g, std::vector<int32_t>* src) const {
  const std::vector<int32_t> slabs = borrowed_slabs();
  const int32_t m = int32_t(slabs.size()), k = cfg_.group, S = cfg_.slab_blocks;
  src->assign(size_t(m) * k * S, -1);
  for (int32_t r = 0; r < m; ++r)
    for (int32_t j = 0; j < k; ++j)
      for (int32_t p = 0; p < S; ++p)
        (*src)[size_t(stage_index(r, m, j, p))] =
            int32_t(n_local_ + slab_slot(slabs[r], g * k + j, p));
}

void SliceBook::set_pos(int32_t pos, int32_t o) {
  const int32_t S = cfg_.slab_blocks;
  const int32_t i = pos / S, p = pos - i * S;
  const bool was = pos_owner_[pos] != kFree, is = o != kFree;
  pos_owner_[pos] = o;
  slab_used_[i] += int32_t(is) - int32_t(was);
  for (int32_t l = 0; l < cfg_.layers; ++l) set_owner(int32_t(n_local_ + slab_slot(i, l, p)), o);
}

void SliceBook::set_slab(int32_t i, int32_t tag) {
  const int32_t S = cfg_.slab_blocks;
  const int32_t t = tag == kLender ? kLender : kFree;
  if ((slab_tag_[i] == kBorrowed) != (tag == kBorrowed)) ++slab_version_;
  slab_tag_[i] = tag;
  for (int32_t p = 0; p < S; ++p) pos_owner_[size_t(i) * S + p] = kFree;
  slab_used_[i] = 0;
  for (int32_t l = 0; l < cfg_.layers; ++l)
    for (int32_t p = 0; p < S; ++p) set_owner(int32_t(n_local_ + slab_slot(i, l, p)), t);
}

void SliceBook::release_if_empty(int32_t i) {
  if (slab_tag_[i] == kBorrowed && slab_used_[i] == 0) set_slab(i, kFree);
}

int SliceBook::slab_init(const SlabCfg& c, std::string* err) {
  if (slab_mode_) {
    *err = "slab_init: the slice is already managed in slabs";
    return kErrInval;
  }
  if (c.layers < 1 || c.slab_blocks < 1 || c.group < 1 || c.layers % c.group ||
      c.layout < 0 || c.layout > 2) {
    *err = "slab_init: layers, slab_blocks and group must be >= 1, group must divide layers, "
           "layout 0..2";
    return kErrInval;
  }
  if (lim_ != n_slice_ || free_slice_.count() != n_slice_) {
    *err = "slab_init: the slice must be untouched (every slot lent and free)";
    return kErrInval;
  }
  const int64_t per = int64_t(c.layers) * c.slab_blocks;
  const int64_t n = n_slice_ / per;
  if (n < 1) {
    *err = "slab_init: the slice holds no whole slab";
    return kErrInval;
  }
  cfg_ = c;
  n_slabs_ = int32_t(n);
  slab_tag_.assign(size_t(n), kFree);
  pos_owner_.assign(size_t(n) * c.slab_blocks, kFree);
  slab_used_.assign(size_t(n), 0);
  slab_mode_ = true;
  ++slab_version_;
  for (int64_t s = n * per; s < n_slice_; ++s) set_owner(int32_t(n_local_ + s), kLender);
  return kOk;
}

int SliceBook::slab_alloc(int32_t n, const int32_t* owners, int32_t* out_pos, std::string* err) {
  if (!slab_mode_) {
    *err = "slab_alloc: the slice is not managed in slabs";
    return kErrInval;
  }
  if (n < 0 || (n > 0 && (!owners || !out_pos))) {
    *err = "slab_alloc: n < 0 or NULL array";
    return kErrInval;
  }
  for (int32_t i = 0; i < n; ++i)
    if (owners[i] < 0) {
      *err = "slab_alloc: slab positions are owned by sequences";
      return kErrInval;
    }
  const int32_t S = cfg_.slab_blocks;
  // free positions of borrowed slabs (index order), then whole free slabs
  std::vector<int32_t> free_pos;
  std::vector<int32_t> free_slabs;
  int64_t room = 0;
  for (int32_t i = 0; i < n_slabs_ && room < n; ++i) {
    if (slab_tag_[i] == kBorrowed && slab_used_[i] < S) room += S - slab_used_[i];
  }
  for (int32_t i = 0; i < n_slabs_ && room < n; ++i)
    if (slab_tag_[i] == kFree) room += S;
  if (room < n) {
    *err = "slab_alloc: not enough slab positions";
    return kErrNomem;
  }
  for (int32_t i = 0; i < n_slabs_ && int64_t(free_pos.size()) < n; ++i)
    if (slab_tag_[i] == kBorrowed && slab_used_[i] < S)
      for (int32_t p = 0; p < S; ++p)
        if (pos_owner_[size_t(i) * S + p] == kFree) free_pos.push_back(i * S + p);
  for (int32_t i = 0; i < n_slabs_; ++i)
    if (slab_tag_[i] == kFree) free_slabs.push_back(i);
  // ---- from here on the book changes ----
  size_t next = 0, next_slab = 0;
  for (int32_t k = 0; k < n; ++k) {
    if (next == free_pos.size()) {
      const int32_t i = free_slabs[next_slab++];
      set_slab(i, kBorrowed);
      for (int32_t p = 0; p < S; ++p) free_pos.push_back(i * S + p);
    }
    const int32_t pos = free_pos[next++];
    set_pos(pos, owners[k]);
    out_pos[k] = pos;
  }
  return kOk;
}

int SliceBook::slab_free(const int32_t* pos, int32_t n, std::string* err) {
  if (!slab_mode_) {
    *err = "slab_free: the slice is not managed in slabs";
    return kErrInval;
  }
  if (n < 0 || (n > 0 && !pos)) {
    *err = "slab_free: n < 0 or NULL array";
    return kErrInval;
  }
  const int64_t n_pos = int64_t(n_slabs_) * cfg_.slab_blocks;
  std::vector<int32_t> sorted(pos, pos + n);
  std::sort(sorted.begin(), sorted.end());
  for (int32_t i = 0; i + 1 < n; ++i)
    if (sorted[i] == sorted[i + 1]) {
      *err = "slab_free: duplicate position";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (pos[i] < 0 || pos[i] >= n_pos) {
      *err = "slab_free: position out of range";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (pos_owner_[pos[i]] < 0) {
      *err = "slab_free: position " + std::to_string(pos[i]) + " not allocated";
      return kErrOwner;
    }
  for (int32_t i = 0; i < n; ++i) set_pos(pos[i], kFree);
  for (int32_t i = 0; i < n; ++i) release_if_empty(pos[i] / cfg_.slab_blocks);
  return kOk;
}

int SliceBook::slab_reclaim(int32_t n, SlabReclaimPlan* plan, std::string* err) {
  if (!slab_mode_) {
    *err = "slab_reclaim: the slice is not managed in slabs";
    return kErrInval;
  }
  if (n < 0) {
    *err = "slab_reclaim: n < 0";
    return kErrInval;
  }
  *plan = SlabReclaimPlan();
  int32_t lent = 0;
  for (int32_t i = 0; i < n_slabs_; ++i) lent += slab_tag_[i] != kLender;
  const int32_t ne = std::min(n, lent);
  plan->reclaimed = ne;
  const int32_t S = cfg_.slab_blocks;
  std::vector<int32_t> reqs;
  for (int32_t t = 0; t < ne; ++t) {
    int32_t take = -1;
    for (int32_t i = n_slabs_ - 1; i >= 0 && take < 0; --i)
      if (slab_tag_[i] == kFree) take = i;
    if (take < 0) {
      // the borrowed slab with the fewest active requests (ties: highest index)
      size_t best = ~size_t(0);
      for (int32_t i = n_slabs_ - 1; i >= 0; --i) {
        if (slab_tag_[i] != kBorrowed) continue;
        reqs.assign(pos_owner_.begin() + size_t(i) * S, pos_owner_.begin() + size_t(i + 1) * S);
        std::sort(reqs.begin(), reqs.end());
        const size_t cnt = size_t(std::unique(reqs.begin(), reqs.end()) - reqs.begin()) -
                           size_t(reqs.front() == kFree);
        if (cnt < best) {
          best = cnt;
          take = i;
        }
      }
      reqs.assign(pos_owner_.begin() + size_t(take) * S, pos_owner_.begin() + size_t(take + 1) * S);
      std::sort(reqs.begin(), reqs.end());
      reqs.erase(std::unique(reqs.begin(), reqs.end()), reqs.end());
      for (int32_t r : reqs) {
        if (r < 0) continue;
        plan->victims.push_back(r);
        // the dependency chain: every block the request holds, local or slab
        for (int32_t u = 0; u < n_local_; ++u)
          if (own_local_[u] == r) {
            set_owner(u, kFree);
            plan->released.push_back(u);
          }
        for (int64_t q = 0; q < int64_t(pos_owner_.size()); ++q)
          if (pos_owner_[q] == r) {
            const int32_t i = int32_t(q / S), p = int32_t(q % S);
            for (int32_t l = 0; l < cfg_.layers; ++l)
              plan->released.push_back(int32_t(n_local_ + slab_slot(i, l, p)));
            set_pos(int32_t(q), kFree);
          }
      }
      for (int32_t i = 0; i < n_slabs_; ++i) release_if_empty(i);
    }
    set_slab(take, kLender);
    plan->slabs.push_back(take);
  }
  std::sort(plan->released.begin(), plan->released.end());
  return kOk;
}

}  // namespace ema
