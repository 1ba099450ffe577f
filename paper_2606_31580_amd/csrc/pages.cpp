// Paged KV bookkeeping (host) and the laser_pages_* C ABI over it.
#include "pages.hpp"

#include <new>

#include "laser.h"
#include "laser_error.h"

namespace laser {

PagePool::PagePool(int num_pages, int page_size, int max_seqs, int max_pages_per_seq)
    : num_pages_(num_pages), page_size_(page_size), max_seqs_(max_seqs), max_pages_per_seq_(max_pages_per_seq),
      tables_(max_seqs), lens_(max_seqs, 0), live_(max_seqs, 0), refs_(num_pages, 0) {
  for (int i = 0; i < num_pages; ++i) free_.insert(free_.end(), i);
}

int PagePool::take_lowest() {
  int p = *free_.begin();
  free_.erase(free_.begin());
  refs_[p] = 1;
  return p;
}

void PagePool::release(int page) {
  if (--refs_[page] == 0) free_.insert(page);
}

int PagePool::add_seq(int seq, int length, std::vector<PageUpdate>* upd) {
  if (seq < 0 || seq >= max_seqs_) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d out of range", seq);
  if (live_[seq]) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d already present", seq);
  if (length < 0) return laser_fail(LASER_ERR_INVALID_ARG, "negative length");
  int need = pages_for(length);
  if (need > max_pages_per_seq_)
    return laser_fail(LASER_ERR_INVALID_ARG, "length %d exceeds max_pages_per_seq", length);
  if (need > (int)free_.size()) return laser_fail(LASER_ERR_OUT_OF_PAGES, "need %d pages, %d free", need, (int)free_.size());
  tables_[seq].clear();
  for (int i = 0; i < need; ++i) {
    int p = take_lowest();
    tables_[seq].push_back(p);
    if (upd) upd->push_back({seq, i, p});
  }
  lens_[seq] = length;
  live_[seq] = 1;
  return LASER_OK;
}

int PagePool::pages_needed(int seq, int n) const {
  return pages_for(lens_[seq] + n) - (int)tables_[seq].size();
}

int PagePool::append(int seq, int n, std::vector<PageUpdate>* upd) {
  if (!live(seq)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq);
  if (n < 0) return laser_fail(LASER_ERR_INVALID_ARG, "negative growth");
  int need = pages_needed(seq, n);
  if (pages_for(lens_[seq] + n) > max_pages_per_seq_)
    return laser_fail(LASER_ERR_INVALID_ARG, "seq %d would exceed max_pages_per_seq", seq);
  if (need > (int)free_.size()) return laser_fail(LASER_ERR_OUT_OF_PAGES, "need %d pages, %d free", need, (int)free_.size());
  for (int i = 0; i < need; ++i) {
    int p = take_lowest();
    if (upd) upd->push_back({seq, (int)tables_[seq].size(), p});
    tables_[seq].push_back(p);
  }
  lens_[seq] += n;
  return LASER_OK;
}

int PagePool::truncate(int seq, int length) {
  if (!live(seq)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq);
  if (length < 0 || length > lens_[seq]) return laser_fail(LASER_ERR_INVALID_ARG, "truncate length out of range");
  int keep = pages_for(length);
  if (length % page_size_ != 0 && refs_[tables_[seq][keep - 1]] > 1)
    return laser_fail(LASER_ERR_INVALID_ARG, "seq %d: length %d ends inside a shared page", seq, length);
  for (size_t i = keep; i < tables_[seq].size(); ++i) release(tables_[seq][i]);
  tables_[seq].resize(keep);
  lens_[seq] = length;
  return LASER_OK;
}

int PagePool::fork(int src, int dst, std::vector<PageUpdate>* upd, PageCopy* copy, bool* has_copy) {
  if (!live(src)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", src);
  if (dst < 0 || dst >= max_seqs_) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d out of range", dst);
  if (live_[dst]) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d already present", dst);
  const int full = lens_[src] / page_size_;
  const bool partial = lens_[src] % page_size_ != 0;
  if (partial && free_.empty()) return laser_fail(LASER_ERR_OUT_OF_PAGES, "need 1 page, 0 free");
  tables_[dst].clear();
  for (int i = 0; i < full; ++i) {
    const int p = tables_[src][i];
    ++refs_[p];
    tables_[dst].push_back(p);
    if (upd) upd->push_back({dst, i, p});
  }
  *has_copy = partial;
  if (partial) {
    const int p = take_lowest();
    copy->src = tables_[src][full];
    copy->dst = p;
    tables_[dst].push_back(p);
    if (upd) upd->push_back({dst, full, p});
  }
  lens_[dst] = lens_[src];
  live_[dst] = 1;
  return LASER_OK;
}

int PagePool::free_seq(int seq) {
  if (!live(seq)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq);
  truncate(seq, 0);
  live_[seq] = 0;
  return LASER_OK;
}

}  // namespace laser

struct laser_page_pool {
  unsigned magic;
  laser::PagePool pool;
};

static const unsigned kPoolMagic = 0x50414745u;

static laser::PagePool* get_pool(const laser_page_pool* p) {
  if (!p || p->magic != kPoolMagic) return nullptr;
  return const_cast<laser::PagePool*>(&p->pool);
}

extern "C" {

laser_status laser_pages_create(int num_pages, int page_size, int max_seqs, int max_pages_per_seq,
                                laser_page_pool** out) {
  if (!out) return laser_fail(LASER_ERR_INVALID_ARG, "out is NULL");
  if (num_pages < 1 || page_size < 1 || max_seqs < 1 || max_pages_per_seq < 1)
    return laser_fail(LASER_ERR_INVALID_ARG, "sizes must be positive");
  auto* h = new (std::nothrow) laser_page_pool{kPoolMagic, laser::PagePool(num_pages, page_size, max_seqs, max_pages_per_seq)};
  if (!h) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  *out = h;
  return LASER_OK;
}

#define POOL_OR_FAIL(h)                                                        \
  laser::PagePool* P = get_pool(h);                                            \
  if (!P) return laser_fail(LASER_ERR_STATE, "invalid or destroyed page pool")

laser_status laser_pages_add_seq(laser_page_pool* h, int seq_id, int length) {
  POOL_OR_FAIL(h);
  return (laser_status)P->add_seq(seq_id, length, nullptr);
}

laser_status laser_pages_append(laser_page_pool* h, int seq_id, int n_tokens) {
  POOL_OR_FAIL(h);
  return (laser_status)P->append(seq_id, n_tokens, nullptr);
}

laser_status laser_pages_truncate(laser_page_pool* h, int seq_id, int length) {
  POOL_OR_FAIL(h);
  return (laser_status)P->truncate(seq_id, length);
}

laser_status laser_pages_fork(laser_page_pool* h, int src_seq, int dst_seq) {
  POOL_OR_FAIL(h);
  laser::PageCopy c{};
  bool has = false;
  return (laser_status)P->fork(src_seq, dst_seq, nullptr, &c, &has);
}

laser_status laser_pages_free_seq(laser_page_pool* h, int seq_id) {
  POOL_OR_FAIL(h);
  return (laser_status)P->free_seq(seq_id);
}

laser_status laser_pages_table(const laser_page_pool* h, int seq_id, int32_t* out, int cap, int* n_out) {
  POOL_OR_FAIL(h);
  if (!out || !n_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!P->live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  const auto& t = P->table(seq_id);
  if ((int)t.size() > cap) return laser_fail(LASER_ERR_INVALID_ARG, "cap %d < %d pages", cap, (int)t.size());
  for (size_t i = 0; i < t.size(); ++i) out[i] = t[i];
  *n_out = (int)t.size();
  return LASER_OK;
}

laser_status laser_pages_seq_len(const laser_page_pool* h, int seq_id, int* len_out) {
  POOL_OR_FAIL(h);
  if (!len_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!P->live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  *len_out = P->len(seq_id);
  return LASER_OK;
}

laser_status laser_pages_num_free(const laser_page_pool* h, int* n_out) {
  POOL_OR_FAIL(h);
  if (!n_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  *n_out = P->num_free();
  return LASER_OK;
}

laser_status laser_pages_destroy(laser_page_pool* h) {
  POOL_OR_FAIL(h);
  (void)P;
  h->magic = 0;
  delete h;
  return LASER_OK;
}

}  // extern "C"
