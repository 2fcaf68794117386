// Host bookkeeping of the memory slice: see slice_book.h.
#include "slice_book.h"

#include <algorithm>
#include <functional>
#include <unordered_map>
#include <unordered_set>

namespace ema {

// ---------------------------------------------------------------- FreeBits --
void FreeBits::reset(int32_t n, bool all_free) {
  n_ = n;
  w_.assign((size_t(n) + 63) / 64, 0ull);
  count_ = 0;
  if (all_free)
    for (int32_t i = 0; i < n; ++i) set(i, true);
}

void FreeBits::set(int32_t i, bool is_free) {
  uint64_t& w = w_[i >> 6];
  const uint64_t bit = 1ull << (i & 63);
  const bool was = (w & bit) != 0;
  if (was == is_free) return;
  if (is_free) {
    w |= bit;
    ++count_;
  } else {
    w &= ~bit;
    --count_;
  }
}

int32_t FreeBits::lowest(int32_t k, int32_t limit, int32_t* out) const {
  int32_t got = 0;
  limit = std::min(limit, n_);
  for (size_t wi = 0; got < k && int64_t(wi) * 64 < limit; ++wi) {
    uint64_t w = w_[wi];
    while (w && got < k) {
      const int32_t b = __builtin_ctzll(w);
      const int32_t i = int32_t(wi * 64 + b);
      if (i >= limit) return got;
      out[got++] = i;
      w &= w - 1;
    }
  }
  return got;
}

int32_t FreeBits::count_below(int32_t limit) const {
  limit = std::min(limit, n_);
  int32_t c = 0;
  const int32_t full = limit >> 6;
  for (int32_t wi = 0; wi < full; ++wi) c += __builtin_popcountll(w_[wi]);
  const int32_t rem = limit & 63;
  if (rem) c += __builtin_popcountll(w_[full] & ((1ull << rem) - 1));
  return c;
}

// --------------------------------------------------------------- SliceBook --
void SliceBook::init(int32_t n_local, int32_t n_slice) {
  n_local_ = n_local;
  n_slice_ = n_slice;
  lim_ = n_slice;
  own_local_.assign(n_local, kFree);
  own_slice_.assign(n_slice, kFree);
  free_local_.reset(n_local, true);
  free_slice_.reset(n_slice, true);
}

void SliceBook::set_owner(int32_t u, int32_t o) {
  if (u < n_local_) {
    own_local_[u] = o;
    free_local_.set(u, o == kFree);
  } else {
    const int32_t s = u - n_local_;
    own_slice_[s] = o;
    free_slice_.set(s, o == kFree);
  }
}

int SliceBook::alloc(int32_t pool, int32_t n, const int32_t* owners, int32_t* out_ids,
                     std::string* err) {
  if (n < 0 || (n > 0 && (!owners || !out_ids))) {
    *err = "alloc: n < 0 or NULL array";
    return kErrInval;
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t o = owners[i];
    if (o < 0 && o != kStaging) {
      *err = "alloc: bad owner " + std::to_string(o);
      return kErrInval;
    }
    if (o == kStaging && pool != 0) {
      *err = "alloc: staging blocks are local";
      return kErrInval;
    }
  }
  if (pool != 0 && pool != 1) {
    *err = "alloc: bad pool";
    return kErrInval;
  }
  if (pool == 1 && slab_mode_) {
    *err = "alloc: the slice is managed in slabs (slab_alloc)";
    return kErrInval;
  }
  FreeBits& fb = pool == 0 ? free_local_ : free_slice_;
  const int32_t limit = pool == 0 ? n_local_ : lim_;
  if (fb.count_below(limit) < n) {
    *err = "alloc: not enough free blocks";
    return kErrNomem;
  }
  std::vector<int32_t> slots(n);
  const int32_t got = fb.lowest(n, limit, slots.data());
  if (got != n) {
    *err = "alloc: internal free-count mismatch";
    return kErrNomem;
  }
  const int32_t base = pool == 0 ? 0 : n_local_;
  for (int32_t i = 0; i < n; ++i) {
    out_ids[i] = base + slots[i];
    set_owner(base + slots[i], owners[i]);
  }
  return kOk;
}

int SliceBook::free_blocks(const int32_t* ids, int32_t n, std::string* err) {
  if (n < 0 || (n > 0 && !ids)) {
    *err = "free: n < 0 or NULL array";
    return kErrInval;
  }
  std::unordered_set<int32_t> seen;
  seen.reserve(size_t(n) * 2);
  for (int32_t i = 0; i < n; ++i)
    if (!seen.insert(ids[i]).second) {
      *err = "free: duplicate id";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (slab_mode_ && ids[i] >= n_local_) {
      *err = "free: the slice is managed in slabs (slab_free)";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i) {
    if (!in_range(ids[i])) {
      *err = "free: id out of range";
      return kErrInval;
    }
    const int32_t o = owner(ids[i]);
    if (o == kFree || o == kLender) {
      *err = "free: block " + std::to_string(ids[i]) + " not allocated";
      return kErrOwner;
    }
  }
  for (int32_t i = 0; i < n; ++i) set_owner(ids[i], kFree);
  return kOk;
}

int SliceBook::lend(int32_t n, int32_t* added, std::string* err) {
  if (n < 0) {
    *err = "lend: n < 0";
    return kErrInval;
  }
  if (slab_mode_) {   // the lowest-indexed lender's slabs
    int32_t got = 0;
    for (int32_t i = 0; i < n_slabs_ && got < n; ++i)
      if (slab_tag_[i] == kLender) {
        set_slab(i, kFree);
        ++got;
      }
    if (added) *added = got;
    return kOk;
  }
  const int32_t nw = int32_t(std::min<int64_t>(n_slice_, int64_t(lim_) + n));
  const int32_t old = lim_;
  lim_ = nw;  // set first so the new slots count as lendable
  for (int32_t s = old; s < nw; ++s) set_owner(n_local_ + s, kFree);
  if (added) *added = nw - old;
  return kOk;
}

int SliceBook::check_pairs(const int32_t* src, const int32_t* dst, int32_t n,
                           std::string* err) const {
  if (n < 0 || (n > 0 && (!src || !dst))) {
    *err = "copy list: n < 0 or NULL array";
    return kErrInval;
  }
  std::unordered_set<int32_t> d;
  d.reserve(size_t(n) * 2);
  for (int32_t i = 0; i < n; ++i)
    if (!d.insert(dst[i]).second) {
      *err = "copy list: duplicate destination";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (d.count(src[i])) {
      *err = "copy list: source and destination overlap";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (!in_range(src[i]) || !in_range(dst[i])) {
      *err = "copy list: id out of range";
      return kErrInval;
    }
  return kOk;
}

int SliceBook::check_prefetch(const int32_t* src, const int32_t* dst, int32_t n,
                              std::string* err) const {
  int rc = check_pairs(src, dst, n, err);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i)
    if (src[i] < n_local_ || owner(src[i]) < 0) {
      *err = "prefetch: source " + std::to_string(src[i]) + " is not an owned slice block";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (dst[i] >= n_local_ || owner(dst[i]) != kStaging) {
      *err = "prefetch: destination " + std::to_string(dst[i]) + " is not a staging block";
      return kErrInval;
    }
  return kOk;
}

int SliceBook::check_migrate(const int32_t* src, const int32_t* dst, int32_t n,
                             std::string* err) const {
  int rc = check_pairs(src, dst, n, err);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t o = owner(src[i]);
    if (o < 0 || owner(dst[i]) != o) {
      *err = "migrate: owners differ or source unowned";
      return kErrInval;
    }
  }
  return kOk;
}

int SliceBook::check_writeback(const int32_t* src, const int32_t* dst, int32_t n,
                               std::string* err) const {
  int rc = check_pairs(src, dst, n, err);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i)
    if (src[i] >= n_local_ || owner(src[i]) != kStaging) {
      *err = "writeback: source " + std::to_string(src[i]) + " is not a staging block";
      return kErrInval;
    }
  for (int32_t i = 0; i < n; ++i)
    if (dst[i] < n_local_ || owner(dst[i]) < 0) {
      *err = "writeback: destination " + std::to_string(dst[i]) + " is not an owned slice block";
      return kErrInval;
    }
  return kOk;
}

int SliceBook::reclaim(int32_t n, ReclaimPlan* p, std::string* err) {
  if (n < 0) {
    *err = "reclaim: n < 0";
    return kErrInval;
  }
  if (slab_mode_) {
    *err = "reclaim: the slice is managed in slabs (slab_reclaim)";
    return kErrInval;
  }
  *p = ReclaimPlan();
  const int32_t ne = std::min(n, lim_);
  const int32_t cut = lim_ - ne;
  p->reclaimed = ne;
  p->cut = cut;

  // Every allocation comes before the first change of state, so a failed
  // host allocation leaves the book as it was.
  std::vector<int32_t> movers;  // slice slots in [cut, lim) owned by a sequence
  movers.reserve(size_t(ne));
  for (int32_t s = cut; s < lim_; ++s)
    if (own_slice_[s] >= 0) movers.push_back(s);
  const size_t m0 = movers.size();
  auto n_dest = [&]() {
    return int64_t(free_slice_.count_below(cut)) + free_local_.count();
  };
  // Preempting an owner removes only its own movers, so the owners ranked
  // once by (movers desc, id desc) give the order in which step 4 takes them,
  // and each preemption adds the owner's local blocks and its slice blocks
  // below the cut to the destinations: the victims follow from counts alone.
  std::vector<std::vector<int32_t>> held;      // blocks of each victim, ascending
  if (int64_t(m0) > n_dest()) {
    std::vector<int32_t> own(m0);
    for (size_t i = 0; i < m0; ++i) own[i] = own_slice_[movers[i]];
    std::sort(own.begin(), own.end());
    std::vector<std::pair<int32_t, int32_t>> rank;   // (movers, owner)
    for (size_t i = 0; i < m0;) {
      size_t j = i;
      while (j < m0 && own[j] == own[i]) ++j;
      rank.emplace_back(int32_t(j - i), own[i]);
      i = j;
    }
    std::sort(rank.begin(), rank.end(), std::greater<std::pair<int32_t, int32_t>>());
    std::unordered_map<int32_t, size_t> pos;         // owner -> rank position
    pos.reserve(rank.size() * 2);
    for (size_t k = 0; k < rank.size(); ++k) pos[rank[k].second] = k;
    std::vector<int64_t> frees(rank.size(), 0);      // destinations its preemption adds
    for (int32_t u = 0; u < n_local_; ++u) {
      auto it = own_local_[u] >= 0 ? pos.find(own_local_[u]) : pos.end();
      if (it != pos.end()) ++frees[it->second];
    }
    for (int32_t s = 0; s < cut; ++s) {
      auto it = own_slice_[s] >= 0 ? pos.find(own_slice_[s]) : pos.end();
      if (it != pos.end()) ++frees[it->second];
    }
    int64_t alive = int64_t(m0), dest = n_dest();
    size_t nv = 0;
    while (alive > dest) {
      alive -= rank[nv].first;
      dest += frees[nv];
      ++nv;
    }
    held.resize(nv);
    for (int32_t u = 0; u < n_local_ + n_slice_; ++u) {
      const int32_t o = u < n_local_ ? own_local_[u] : own_slice_[u - n_local_];
      auto it = o >= 0 ? pos.find(o) : pos.end();
      if (it != pos.end() && it->second < nv) held[it->second].push_back(u);
    }
    p->victims.reserve(nv);
    size_t total = 0;
    for (const auto& v : held) total += v.size();
    p->victim_blocks.reserve(total);
    for (size_t k = 0; k < nv; ++k) p->victims.push_back(rank[k].second);
  }
  std::vector<int32_t> dst(m0);
  p->move_src.reserve(m0);
  p->move_dst.reserve(m0);

  // ---- from here on the book changes and nothing allocates ----
  for (const auto& blocks : held)
    for (int32_t u : blocks) {
      p->victim_blocks.push_back(u);
      set_owner(u, kFree);
    }
  if (!p->victims.empty())
    movers.erase(std::remove_if(movers.begin(), movers.end(),
                                [&](int32_t s) { return own_slice_[s] < 0; }),
                 movers.end());

  const int32_t m = int32_t(movers.size());
  const int32_t got_s = free_slice_.lowest(m, cut, dst.data());
  for (int32_t i = 0; i < got_s; ++i) dst[i] += n_local_;
  const int32_t got_l = free_local_.lowest(m - got_s, n_local_, dst.data() + got_s);
  // got_s + got_l == m: the victims were chosen so that m <= n_dest()
  for (int32_t i = 0; i < m; ++i) {
    const int32_t o = own_slice_[movers[i]];
    p->move_src.push_back(n_local_ + movers[i]);
    p->move_dst.push_back(dst[i]);
    set_owner(dst[i], o);
  }
  p->written_back = got_l;
  for (int32_t s = cut; s < lim_; ++s) set_owner(n_local_ + s, kLender);
  lim_ = cut;
  return kOk;
}

}  // namespace ema
