// Continuous batching with preemption, on top of the waiting queue.
//
// One engine iteration ("step") at time now:
//   1. every running request will decode one token this step; if the KV pool
//      cannot hold that many positions, running requests are preempted until
//      it can -- SJF evicts the largest estimated job, HRRN the lowest current
//      response ratio (the preemption rule of the paper's implementation
//      appendix), FCFS the most recently admitted one (the serving engines'
//      recompute-on-preemption default).  A preempted request drops its
//      generated tokens and returns to the waiting queue with its original
//      arrival time and keys;
//   2. free slots are refilled from the queue in the policy's order (each
//      admitted request is prefilled this step and produces its first token
//      in it), stopping at the first request the pool cannot hold, at the
//      per-step admission limit, or when no slot is free;
//   3. the decode rows are the surviving running requests (admission order)
//      followed by the admitted ones (not those, with defer_first: they then
//      start decoding in the next step); after the step each row has one more
//      token and a request leaves when it reaches its token count.
//
// KV pool accounting (in token positions): a running request holds
// cross_tokens (its cross-attention cache) plus one position per generated
// token.  kv_capacity <= 0 disables the pool limit (slots alone bound the
// batch).  Everything is integer and depends only on the inputs, so a run is
// reproducible step for step.
#pragma once

#include <stdint.h>

#include <vector>

#include "queue.h"

namespace asr {

struct ServeConfig {
  int32_t n_slots = 0;         // usable slots (<= physical slots and decode rows)
  int32_t max_admit = 0;       // admissions per step
  int64_t kv_capacity = 0;     // pool size in token positions; <= 0: unlimited
  int32_t cross_tokens = 0;    // positions charged for a request's cross cache
  int32_t tok_num = 27, tok_den = 10;   // output tokens per audio-second (rational)
  int32_t start_token = 0;     // decoder input at position 0
  // dynamic policy switching (0: the queue's policy throughout)
  int32_t dynamic = 0;
  int32_t depth_low = 0;       // eligible waiting <= depth_low: FCFS
  int64_t starve_num = 0, starve_den = 1;   // some ratio above this: HRRN, else SJF
  // admitted requests produce their first token in the step after the one
  // that prefills them (so a step's prefill and its decode rows are independent)
  int32_t defer_first = 0;
};

struct RunEntry {
  QEntry q;                    // queue record (keys, samples, max_tokens)
  int32_t slot = -1;
  int32_t generated = 0;       // tokens produced so far (= self-cache positions held)
  int32_t total = 0;           // tokens to produce
  int64_t admit_seq = 0;       // admission order
  int32_t last_token = 0;      // input of the next decode step
  std::vector<int32_t> tokens;
};

struct ServePlan {
  int32_t policy = 0;                     // policy the step ran under
  std::vector<int64_t> preempted;
  std::vector<int64_t> admitted;          // ids, prefilled this step
  std::vector<int32_t> admitted_slot;
  // decode rows of this step
  std::vector<int64_t> dec_id;
  std::vector<int32_t> dec_slot, dec_pos, dec_token;
};

class ServeEngine {
 public:
  void configure(const ServeConfig& c);
  const ServeConfig& config() const { return cfg_; }
  bool busy() const { return !run_.empty(); }
  int running() const { return (int)run_.size(); }
  int64_t kv_used() const;

  // Tokens a request produces: round-half-up of duration * rate, clamped to
  // [1, min(448, max_tokens)].
  int32_t tokens_for(const QEntry& e) const;

  // Decide one step (preempted requests go back into q after admission, so
  // none is re-admitted in the step that evicted it).  The plan's decode rows
  // are in the order the step's outputs must be committed.
  ServePlan plan(int64_t now_us, WaitQueue& q);

  // Apply a step's outputs: tokens[i] is the token produced by decode row i
  // (NULL when no model ran: tokens are recorded as -1).  Returns the ids
  // that finished; gen_after (optional) receives each decode row's token
  // count after the step.
  std::vector<int64_t> commit(const ServePlan& p, const int32_t* tokens,
                              std::vector<int32_t>* gen_after = nullptr);

  // Tokens of a finished request (once), false when unknown.
  bool take_result(int64_t id, std::vector<int32_t>* tokens);
  bool has_result(int64_t id) const;
  const RunEntry* find(int64_t id) const;
  int64_t steps_under(int policy) const { return steps_by_policy_[policy]; }

  // The dynamic rule: FCFS while at most depth_low requests wait (every one
  // of them is about to be admitted anyway, so arrival order costs nothing);
  // otherwise HRRN as soon as some waiting request's response ratio exceeds
  // the starvation threshold, else SJF.
  int choose_policy(int64_t now_us, const WaitQueue& q) const;

 private:
  // true when running entry a is evicted before b at time now
  bool worse(const RunEntry& a, const RunEntry& b, int64_t now_us, int policy) const;

  ServeConfig cfg_;
  std::vector<RunEntry> run_;                 // admission order
  std::vector<int32_t> free_slots_;
  int64_t seq_ = 0;
  int64_t steps_by_policy_[3] = {0, 0, 0};
  std::vector<std::pair<int64_t, std::vector<int32_t>>> done_;
};

}  // namespace asr
