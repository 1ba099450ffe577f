// Host bookkeeping of the paged KV cache: fixed-size pages handed out by lowest free id.
#pragma once

#include <cstdint>
#include <set>
#include <vector>

namespace laser {

struct PageUpdate {
  int seq, idx, page;  // block_table[seq][idx] = page
};

// A page whose contents must be copied to another page (the partial last page of a fork).
struct PageCopy {
  int src, dst;
};

class PagePool {
 public:
  PagePool(int num_pages, int page_size, int max_seqs, int max_pages_per_seq);

  int num_pages() const { return num_pages_; }
  int page_size() const { return page_size_; }
  int max_seqs() const { return max_seqs_; }
  int max_pages_per_seq() const { return max_pages_per_seq_; }
  int num_free() const { return (int)free_.size(); }
  bool live(int seq) const { return seq >= 0 && seq < max_seqs_ && live_[seq]; }
  int len(int seq) const { return lens_[seq]; }
  const std::vector<int>& table(int seq) const { return tables_[seq]; }
  int pages_for(int n) const { return (n + page_size_ - 1) / page_size_; }

  // All of these validate first and change nothing when they fail (laser_status codes).
  int add_seq(int seq, int length, std::vector<PageUpdate>* upd);
  // Pages a growth of n tokens would take (0 if it fits in the current last page).
  int pages_needed(int seq, int n) const;
  int append(int seq, int n, std::vector<PageUpdate>* upd);
  int truncate(int seq, int length);
  int free_seq(int seq);
  // dst (a free slot) sees src's current positions: src's full pages are shared (reference
  // counted), the page holding the partial tail (if any) is copied into a fresh page.
  int fork(int src, int dst, std::vector<PageUpdate>* upd, PageCopy* copy, bool* has_copy);
  int refs(int page) const { return refs_[page]; }

 private:
  int take_lowest();
  void release(int page);
  int num_pages_, page_size_, max_seqs_, max_pages_per_seq_;
  std::set<int> free_;
  std::vector<std::vector<int>> tables_;
  std::vector<int> lens_;
  std::vector<char> live_;
  std::vector<int> refs_;  // tables referencing each page
};

}  // namespace laser
