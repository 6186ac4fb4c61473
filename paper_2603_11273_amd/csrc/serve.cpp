#include "serve.h"

#include <algorithm>

namespace asr {

void ServeEngine::configure(const ServeConfig& c) {
  cfg_ = c;
  run_.clear();
  done_.clear();
  seq_ = 0;
  free_slots_.clear();
  for (int s = 0; s < cfg_.n_slots; ++s) free_slots_.push_back(s);
  steps_by_policy_[0] = steps_by_policy_[1] = steps_by_policy_[2] = 0;
}

int64_t ServeEngine::kv_used() const {
  int64_t u = 0;
  for (const auto& r : run_) u += cfg_.cross_tokens + r.generated;
  return u;
}

int32_t ServeEngine::tokens_for(const QEntry& e) const {
  // round-half-up(n * num / (sr * den)) = floor((2 n num + sr den) / (2 sr den))
  const int64_t den = (int64_t)e.sample_rate * cfg_.tok_den;
  int64_t t = (2 * e.n_samples * (int64_t)cfg_.tok_num + den) / (2 * den);
  const int64_t cap = std::min<int64_t>(448, e.max_tokens > 0 ? e.max_tokens : 448);
  if (t > cap) t = cap;
  if (t < 1) t = 1;
  return (int32_t)t;
}

bool ServeEngine::worse(const RunEntry& a, const RunEntry& b, int64_t now_us, int policy) const {
  if (policy == WaitQueue::FCFS) {
    if (a.admit_seq != b.admit_seq) return a.admit_seq > b.admit_seq;
    return a.q.id > b.q.id;
  }
  if (policy == WaitQueue::HRRN) {
    // R_a < R_b  <=>  (w_a + e_a) e_b < (w_b + e_b) e_a  <=>  w_a e_b < w_b e_a
    const __int128 lhs = (__int128)(now_us - a.q.arrival_us) * b.q.job;
    const __int128 rhs = (__int128)(now_us - b.q.arrival_us) * a.q.job;
    if (lhs != rhs) return lhs < rhs;
  }
  // SJF order reversed: largest job, then latest arrival, then largest id
  if (a.q.job != b.q.job) return a.q.job > b.q.job;
  if (a.q.arrival_us != b.q.arrival_us) return a.q.arrival_us > b.q.arrival_us;
  return a.q.id > b.q.id;
}

int ServeEngine::choose_policy(int64_t now_us, const WaitQueue& q) const {
  if (q.eligible_count(now_us) <= cfg_.depth_low) return WaitQueue::FCFS;
  int64_t n = 0, d = 1;
  q.max_ratio(now_us, &n, &d);
  // n / d > starve_num / starve_den
  if ((__int128)n * cfg_.starve_den > (__int128)cfg_.starve_num * d) return WaitQueue::HRRN;
  return WaitQueue::SJF;
}

ServePlan ServeEngine::plan(int64_t now_us, WaitQueue& q) {
  ServePlan p;
  if (cfg_.dynamic) {
    const int want = choose_policy(now_us, q);
    if (want != q.policy()) q.set_policy(want, q.kappa_num(), q.kappa_den());
  }
  const int policy = q.policy();
  p.policy = policy;
  steps_by_policy_[policy] += 1;
  const bool limited = cfg_.kv_capacity > 0;
  // 1. every running request grows by one position this step
  int64_t need = 0;
  for (const auto& r : run_) need += cfg_.cross_tokens + r.generated + 1;
  std::vector<QEntry> requeue;
  while (limited && need > cfg_.kv_capacity && !run_.empty()) {
    size_t v = 0;
    for (size_t i = 1; i < run_.size(); ++i)
      if (worse(run_[i], run_[v], now_us, policy)) v = i;
    need -= cfg_.cross_tokens + run_[v].generated + 1;
    p.preempted.push_back(run_[v].q.id);
    requeue.push_back(run_[v].q);
    free_slots_.push_back(run_[v].slot);
    run_.erase(run_.begin() + (long)v);
  }
  std::sort(free_slots_.begin(), free_slots_.end());
  // 2. admissions in policy order
  while ((int)p.admitted.size() < cfg_.max_admit && !free_slots_.empty()) {
    if (limited && need + cfg_.cross_tokens + 1 > cfg_.kv_capacity) break;
    std::vector<QEntry> got = q.pop_batch(now_us, 1);
    if (got.empty()) break;
    RunEntry r;
    r.q = got[0];
    r.slot = free_slots_.front();
    free_slots_.erase(free_slots_.begin());
    r.total = tokens_for(r.q);
    r.admit_seq = seq_++;
    r.last_token = cfg_.start_token;
    need += cfg_.cross_tokens + 1;
    p.admitted.push_back(r.q.id);
    p.admitted_slot.push_back(r.slot);
    run_.push_back(std::move(r));
  }
  for (auto& e : requeue) q.push(e);
  // 3. decode rows: everything running, in admission order (with defer_first
  //    the requests admitted in this step wait for the next one)
  const size_t n_rows = cfg_.defer_first ? run_.size() - p.admitted.size() : run_.size();
  for (size_t i = 0; i < n_rows; ++i) {
    const RunEntry& r = run_[i];
    p.dec_id.push_back(r.q.id);
    p.dec_slot.push_back(r.slot);
    p.dec_pos.push_back(r.generated);
    p.dec_token.push_back(r.generated == 0 ? cfg_.start_token : r.last_token);
  }
  return p;
}

std::vector<int64_t> ServeEngine::commit(const ServePlan& p, const int32_t* tokens,
                                         std::vector<int32_t>* gen_after) {
  std::vector<int64_t> finished;
  if (gen_after) gen_after->assign(p.dec_id.size(), 0);
  for (size_t i = 0; i < p.dec_id.size(); ++i) {
    // running entries are in the plan's order; find by id to stay robust
    auto it = std::find_if(run_.begin(), run_.end(),
                           [&](const RunEntry& r) { return r.q.id == p.dec_id[i]; });
    if (it == run_.end()) continue;
    const int32_t t = tokens ? tokens[i] : -1;
    it->tokens.push_back(t);
    it->last_token = t;
    it->generated += 1;
    if (gen_after) (*gen_after)[i] = it->generated;
  }
  for (size_t i = 0; i < run_.size();) {
    if (run_[i].generated >= run_[i].total) {
      finished.push_back(run_[i].q.id);
      free_slots_.push_back(run_[i].slot);
      done_.emplace_back(run_[i].q.id, std::move(run_[i].tokens));
      run_.erase(run_.begin() + (long)i);
    } else {
      ++i;
    }
  }
  std::sort(free_slots_.begin(), free_slots_.end());
  return finished;
}

bool ServeEngine::has_result(int64_t id) const {
  for (const auto& d : done_)
    if (d.first == id) return true;
  return false;
}

bool ServeEngine::take_result(int64_t id, std::vector<int32_t>* tokens) {
  for (size_t i = 0; i < done_.size(); ++i)
    if (done_[i].first == id) {
      if (tokens) *tokens = std::move(done_[i].second);
      done_.erase(done_.begin() + (long)i);
      return true;
    }
  return false;
}

const RunEntry* ServeEngine::find(int64_t id) const {
  for (const auto& r : run_)
    if (r.q.id == id) return &r;
  return nullptr;
}

}  // namespace asr
