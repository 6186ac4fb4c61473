#include "queue.h"

#include <algorithm>

namespace asr {

int64_t WaitQueue::job_of(const QEntry& e) const {
  if (kd_ == 0) return e.dur_us;
  if (e.n_samples <= 0) return e.max_tokens;                 // request-level fallback
  int64_t est = (e.n_samples * (int64_t)kn_) / ((int64_t)e.sample_rate * kd_);
  return est < 1 ? 1 : est;
}

// True when a is served before b.
bool WaitQueue::before(const QEntry& a, const QEntry& b, int64_t now_us) const {
  if (policy_ == HRRN) {
    // (w_a + e_a)/e_a > (w_b + e_b)/e_b  <=>  w_a * e_b > w_b * e_a
    __int128 lhs = (__int128)(now_us - a.arrival_us) * b.job;
    __int128 rhs = (__int128)(now_us - b.arrival_us) * a.job;
    if (lhs != rhs) return lhs > rhs;
  }
  if (policy_ != FCFS && a.job != b.job) return a.job < b.job;
  if (a.arrival_us != b.arrival_us) return a.arrival_us < b.arrival_us;
  return a.id < b.id;
}

namespace {
bool arrives_after(const QEntry& x, const QEntry& y) {
  if (x.arrival_us != y.arrival_us) return x.arrival_us > y.arrival_us;
  return x.id > y.id;
}
}  // namespace

void WaitQueue::admit_arrived(int64_t now_us) {
  auto cmp = [this](const QEntry& x, const QEntry& y) { return before(y, x, 0); };
  while (!later_.empty() && later_.front().arrival_us <= now_us) {
    std::pop_heap(later_.begin(), later_.end(), arrives_after);
    items_.push_back(later_.back());
    later_.pop_back();
    if (policy_ != HRRN) std::push_heap(items_.begin(), items_.end(), cmp);
  }
}

void WaitQueue::rebuild() {
  // Requests that have not arrived stay in the arrival heap: a policy switch
  // re-keys them but does not move them into the policy's structure.
  for (auto& e : items_) e.job = job_of(e);
  for (auto& e : later_) e.job = job_of(e);
  if (policy_ != HRRN)
    std::make_heap(items_.begin(), items_.end(),
                   [this](const QEntry& x, const QEntry& y) { return before(y, x, 0); });
}

void WaitQueue::set_policy(int policy, int32_t kappa_num, int32_t kappa_den) {
  policy_ = policy;
  kn_ = kappa_num;
  kd_ = kappa_den;
  rebuild();
}

void WaitQueue::push(QEntry e) {
  e.job = job_of(e);
  ids_.insert(e.id);
  later_.push_back(e);
  std::push_heap(later_.begin(), later_.end(), arrives_after);
}

template <typename F>
void WaitQueue::visit_arrived(int64_t now_us, F&& f) const {
  for (const auto& e : items_)
    if (e.arrival_us <= now_us) f(e);
  // later_ is a min-heap by arrival: a node that has not arrived has no
  // arrived descendant, so the walk stops there.
  if (later_.empty() || later_.front().arrival_us > now_us) return;
  std::vector<size_t> stack{0};
  while (!stack.empty()) {
    const size_t i = stack.back();
    stack.pop_back();
    if (later_[i].arrival_us > now_us) continue;
    f(later_[i]);
    if (2 * i + 1 < later_.size()) stack.push_back(2 * i + 1);
    if (2 * i + 2 < later_.size()) stack.push_back(2 * i + 2);
  }
}

std::vector<int64_t> WaitQueue::rank(int64_t now_us) const {
  std::vector<const QEntry*> el;
  visit_arrived(now_us, [&](const QEntry& e) { el.push_back(&e); });
  std::sort(el.begin(), el.end(),
            [&](const QEntry* x, const QEntry* y) { return before(*x, *y, now_us); });
  std::vector<int64_t> ids;
  ids.reserve(el.size());
  for (auto* e : el) ids.push_back(e->id);
  return ids;
}

std::vector<QEntry> WaitQueue::pop_batch(int64_t now_us, int max_n) {
  std::vector<QEntry> out;
  if (max_n <= 0) return out;
  admit_arrived(now_us);
  if (policy_ == HRRN) {
    // ratios depend on now: a linear scan per pop
    while ((int)out.size() < max_n) {
      int best = -1;
      for (int i = 0; i < (int)items_.size(); ++i) {
        if (items_[i].arrival_us > now_us) continue;
        if (best < 0 || before(items_[i], items_[best], now_us)) best = i;
      }
      if (best < 0) break;
      out.push_back(items_[best]);
      items_[best] = items_.back();
      items_.pop_back();
    }
  } else {
    auto cmp = [this](const QEntry& x, const QEntry& y) { return before(y, x, 0); };
    std::vector<QEntry> later;                 // popped but not yet arrived (an earlier now)
    while ((int)out.size() < max_n && !items_.empty()) {
      std::pop_heap(items_.begin(), items_.end(), cmp);
      QEntry e = items_.back();
      items_.pop_back();
      if (e.arrival_us <= now_us) {
        out.push_back(e);
      } else {
        later.push_back(e);
        if (policy_ == FCFS) break;            // arrival order: the rest arrive later still
      }
    }
    for (auto& e : later) {
      items_.push_back(e);
      std::push_heap(items_.begin(), items_.end(), cmp);
    }
  }
  for (auto& e : out) ids_.erase(e.id);
  return out;
}

bool WaitQueue::any_eligible(int64_t now_us) const {
  if (!later_.empty() && later_.front().arrival_us <= now_us) return true;
  for (const auto& e : items_)
    if (e.arrival_us <= now_us) return true;
  return false;
}

int64_t WaitQueue::min_arrival() const {
  int64_t m = later_.empty() ? INT64_MAX : later_.front().arrival_us;
  for (const auto& e : items_) m = std::min(m, e.arrival_us);
  return m;
}

int WaitQueue::eligible_count(int64_t now_us) const {
  int n = 0;
  visit_arrived(now_us, [&](const QEntry&) { ++n; });
  return n;
}

void WaitQueue::max_ratio(int64_t now_us, int64_t* num, int64_t* den) const {
  int64_t bn = 0, bd = 1;
  visit_arrived(now_us, [&](const QEntry& e) {
    const int64_t n = now_us - e.arrival_us + e.job, d = e.job;
    if ((__int128)n * bd > (__int128)bn * d) {
      bn = n;
      bd = d;
    }
  });
  *num = bn;
  *den = bd;
}

}  // namespace asr
