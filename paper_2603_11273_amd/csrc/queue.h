// Host-side waiting queue with FCFS, SJF and HRRN ordering on integer keys.
//
// Section 3.2 of the paper defines the two duration-aware policies: SJF
// serves the shortest job first (earlier arrival first on equal lengths; the
// queue listing of Appendix A.4 keys its min-heap on (estimate, arrival,
// request id)); HRRN serves the highest response ratio
// (wait + job) / job, recomputed at every pop (Appendix A.4).  FCFS is the
// serving engines' default the paper compares against.
//
// Keys are integers: arrival and wait in microseconds, job length in
// microseconds of audio (or Eq. 1 tokens), and HRRN ratios are compared by
// 128-bit cross-multiplication, so orderings are exact and reproducible.
// Equal ratios fall back to the SJF key.  Only requests with
// arrival_us <= now_us are eligible.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <unordered_set>
#include <vector>

namespace asr {

struct QEntry {
  int64_t id;
  int64_t arrival_us;
  int64_t n_samples;
  int64_t dur_us;
  int32_t sample_rate;
  int32_t max_tokens;
  int64_t job;          // job-length key under the current policy
};

class WaitQueue {
 public:
  enum { FCFS = 0, SJF = 1, HRRN = 2 };

  // kappa_den == 0: job = dur_us; otherwise job = max(1, floor(n * kn / (sr * kd))),
  // or max_tokens when the request carries no samples.
  void set_policy(int policy, int32_t kappa_num, int32_t kappa_den);
  int policy() const { return policy_; }
  int32_t kappa_num() const { return kn_; }
  int32_t kappa_den() const { return kd_; }
  // Eligible requests (arrival <= now) and, over them, the largest HRRN
  // response ratio as a fraction (wait + job) / job (0/1 when none).
  int eligible_count(int64_t now_us) const;
  void max_ratio(int64_t now_us, int64_t* num, int64_t* den) const;
  bool contains(int64_t id) const { return ids_.count(id) != 0; }
  size_t size() const { return items_.size() + later_.size(); }
  void push(QEntry e);
  std::vector<int64_t> rank(int64_t now_us) const;
  std::vector<QEntry> pop_batch(int64_t now_us, int max_n);
  bool any_eligible(int64_t now_us) const;
  int64_t min_arrival() const;   // INT64_MAX when empty

 private:
  int64_t job_of(const QEntry& e) const;
  bool before(const QEntry& a, const QEntry& b, int64_t now_us) const;
  void rebuild();

  // Every policy keeps requests that may not have arrived yet in a separate
  // heap by arrival time and moves them into the policy's structure once a
  // pop sees their arrival, so a queue holding many future requests (a
  // simulation submits them all up front) pops, switches policy and scans for
  // eligible requests in time that grows with the arrived ones only.
  void admit_arrived(int64_t now_us);
  template <typename F>
  void visit_arrived(int64_t now_us, F&& f) const;

  int policy_ = FCFS;
  int32_t kn_ = 0, kd_ = 0;
  std::vector<QEntry> items_;   // binary heap under FCFS/SJF, plain list under HRRN
  std::vector<QEntry> later_;   // min-heap by (arrival, id), not yet moved
  std::unordered_set<int64_t> ids_;
};

}  // namespace asr
