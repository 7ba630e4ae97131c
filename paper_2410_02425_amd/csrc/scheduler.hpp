// Continuous-batching scheduler with a maximum-batch-weight budget.
//
// Policy (LLM-Pilot Sec. II-B; the readings of what the paper leaves open):
//  - One running batch of at most max_batch requests; each admitted request
//    reserves in_len + out_len tokens of batch weight until its last token.
//  - Strict FCFS over arrived requests ordered by (arrival, submission order):
//    admission stops at the first request that does not fit (slot, weight,
//    or prompt tokens of one prefill step).  A request takes the lowest free
//    slot.
//  - One iteration = admission, a prefill step over the admitted requests
//    (each yields its first token), then a decode step over all active
//    requests that still owe tokens (rows in slot order, one token each).
//  - Closed loop (Sec. III-C-3 concurrent users, zero think time): the first
//    U requests arrive at time 0; a finished request releases the next
//    unsent one, which arrives at the end of the finishing step and may join
//    at the next iteration.  Open loop: arrivals as given; a request may be
//    admitted once its arrival time is not after the planning time.
// Pure C++ (no HIP): the GPU run loop and the host simulation both drive it.
#pragma once
#include <stdint.h>

#include <algorithm>
#include <vector>

namespace lp {

struct SReq {
  int64_t id = 0;
  int32_t in_len = 0, out_len = 0;
  int64_t arrival_ns = 0;    // open loop: given
  int32_t order = 0;         // submission index
  // run state
  int32_t slot = -1;
  int32_t emitted = 0;
  int64_t arrival_step = -1;  // closed loop: step whose end is the arrival (-1: time 0)
  int state = 0;              // 0 unsent, 1 pending, 2 active, 3 done
  std::vector<int64_t> tok_step;  // global step index that produced each token
};

struct PlanStep {
  int kind = 0;                  // 0 prefill, 1 decode
  std::vector<int32_t> reqs;     // request indices in row order
  std::vector<int32_t> slots;
  std::vector<int32_t> pos;      // decode: position of the fed token; prefill: in_len
  int64_t n_tokens = 0;
  int64_t sum_ctx = 0;           // KV entries after the step, summed over rows
};

class Scheduler {
 public:
  Scheduler(std::vector<SReq> &reqs, int max_batch, int64_t max_weight, int64_t max_prefill,
            bool closed, int concurrency)
      : r_(reqs), max_batch_(max_batch), max_weight_(max_weight), max_prefill_(max_prefill),
        closed_(closed) {
    slot_req_.assign(max_batch, -1);
    for (auto &q : r_) {
      q.slot = -1;
      q.emitted = 0;
      q.arrival_step = -1;
      q.state = 0;
      q.tok_step.clear();
    }
    if (closed) {
      const int u = std::min<int>(concurrency, (int)r_.size());
      for (int i = 0; i < u; ++i) {
        r_[i].state = 1;
        pending_.push_back(i);
      }
      next_unsent_ = u;
    } else {
      for (int i = 0; i < (int)r_.size(); ++i) {
        r_[i].state = 1;
        pending_.push_back(i);
      }
      next_unsent_ = (int)r_.size();
    }
    sort_pending();
  }

  bool finished() const { return done_ == (int)r_.size(); }

  // Open loop with an empty batch: the time the head request arrives (> now),
  // else -1 (there is something to do now).
  int64_t idle_until(int64_t now) const {
    if (closed_ || n_active_ > 0 || pending_.empty()) return -1;
    const int64_t a = r_[pending_.front()].arrival_ns;
    return a > now ? a : -1;
  }

  // Plans one iteration at time `now`.  Steps get global indices step_base,
  // step_base + 1.  Returns the number of steps appended to `out`.
  int plan(int64_t now, int64_t step_base, std::vector<PlanStep> &out) {
    int n_steps = 0;
    std::vector<int32_t> admitted;
    int64_t tokens = 0;
    size_t head = 0;
    while (head < pending_.size()) {
      SReq &q = r_[pending_[head]];
      if (!closed_ && q.arrival_ns > now) break;
      if (n_active_ + (int)admitted.size() >= max_batch_) break;
      if (weight_ + q.in_len + q.out_len > max_weight_) break;
      if (tokens + q.in_len > max_prefill_) break;
      admitted.push_back(pending_[head]);
      tokens += q.in_len;
      weight_ += q.in_len + q.out_len;
      ++head;
    }
    pending_.erase(pending_.begin(), pending_.begin() + head);
    std::vector<std::pair<int32_t, int64_t>> retired;  // (request, finishing step)
    if (!admitted.empty()) {
      PlanStep st;
      st.kind = 0;
      st.n_tokens = tokens;
      const int64_t idx = step_base + n_steps;
      for (int32_t ri : admitted) {
        SReq &q = r_[ri];
        int s = 0;
        while (slot_req_[s] >= 0) ++s;
        slot_req_[s] = ri;
        q.slot = s;
        q.state = 2;
        q.emitted = 1;
        q.tok_step.push_back(idx);
        ++n_active_;
        st.reqs.push_back(ri);
        st.slots.push_back(s);
        st.pos.push_back(q.in_len);
        st.sum_ctx += q.in_len;
      }
      out.push_back(std::move(st));
      ++n_steps;
      for (int32_t ri : admitted)
        if (r_[ri].out_len == 1) retired.push_back({ri, idx});
      for (auto &p : retired) retire(p.first);
    }
    PlanStep dec;
    dec.kind = 1;
    const int64_t didx = step_base + n_steps;
    for (int s = 0; s < max_batch_; ++s) {
      const int32_t ri = slot_req_[s];
      if (ri < 0) continue;
      SReq &q = r_[ri];
      if (q.emitted >= q.out_len) continue;
      dec.reqs.push_back(ri);
      dec.slots.push_back(s);
      dec.pos.push_back(q.in_len + q.emitted - 1);
      dec.sum_ctx += q.in_len + q.emitted;
    }
    if (!dec.reqs.empty()) {
      dec.n_tokens = (int64_t)dec.reqs.size();
      std::vector<int32_t> fin;
      for (int32_t ri : dec.reqs) {
        SReq &q = r_[ri];
        q.emitted += 1;
        q.tok_step.push_back(didx);
        if (q.emitted == q.out_len) fin.push_back(ri);
      }
      out.push_back(std::move(dec));
      ++n_steps;
      for (int32_t ri : fin) {
        retire(ri);
        retired.push_back({ri, didx});
      }
    }
    if (closed_) {
      for (auto &p : retired) {
        if (next_unsent_ < (int)r_.size()) {
          SReq &nq = r_[next_unsent_];
          nq.arrival_step = p.second;
          nq.state = 1;
          pending_.push_back(next_unsent_);
          ++next_unsent_;
        }
      }
    }
    sort_pending();
    return n_steps;
  }

  // Slots freed in the last plan() call are reported through this hook so the
  // engine can return KV blocks.
  std::vector<int32_t> take_retired_slots() {
    std::vector<int32_t> v;
    v.swap(freed_slots_);
    return v;
  }

 private:
  void retire(int32_t ri) {
    SReq &q = r_[ri];
    slot_req_[q.slot] = -1;
    freed_slots_.push_back(q.slot);
    weight_ -= q.in_len + q.out_len;
    q.state = 3;
    --n_active_;
    ++done_;
  }
  void sort_pending() {
    std::stable_sort(pending_.begin(), pending_.end(), [&](int32_t a, int32_t b) {
      const SReq &x = r_[a], &y = r_[b];
      if (closed_) {
        if (x.arrival_step != y.arrival_step) return x.arrival_step < y.arrival_step;
      } else if (x.arrival_ns != y.arrival_ns) {
        return x.arrival_ns < y.arrival_ns;
      }
      return x.order < y.order;
    });
  }

  std::vector<SReq> &r_;
  int max_batch_;
  int64_t max_weight_, max_prefill_;
  bool closed_;
  std::vector<int32_t> pending_;
  std::vector<int32_t> slot_req_;
  std::vector<int32_t> freed_slots_;
  int next_unsent_ = 0;
  int n_active_ = 0;
  int done_ = 0;
  int64_t weight_ = 0;
};

}  // namespace lp
