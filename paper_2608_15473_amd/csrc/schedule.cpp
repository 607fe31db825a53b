// Discrete-event simulation of the layer-wise decode schedule (Q-First, arXiv:2608.15473,
// Appendix D).  Host code; declared in include/qfattn.h.
//
// Every request sweeps its cache once per layer (its attention time a) and, per layer, rides a
// feed-forward pool: a pool serves one departure at a time, a departure takes ffn_time and
// carries every request waiting at that moment, and it leaves only when at least min_batch are
// waiting (or, with a finite max_wait, when the oldest has waited that long).
//   Q-First:  layer l is ready at e_l = max(sweep_l end, ffn_{l-1} return); at e_l the request
//             joins pool l and starts sweep l+1 (e_1 = arrival + a, finish = ffn_L return).
//   Composed: the request joins pool l when sweep l ends; sweep l+1 starts when it returns.
// At each instant all completions (and what they make ready at that same instant) are applied
// before any pool decides whether to depart.  A pool's time-out instant is computed once, by one
// expression (deadline()), both where the wake-up is scheduled and where the departure is
// decided, so the two agree bit for bit for any floating-point times.
#include <math.h>
#include <stdint.h>

#include <deque>
#include <map>
#include <utility>
#include <vector>

#include "qfattn.h"

namespace {

struct Event {
  int kind;   // 0: sweep (r, l) ended; 1: pool l returned `members`
              // (an instant with no events at all is a wake-up for the pools)
  int r, l;
  std::vector<int> members;
};

class Simulation {
 public:
  Simulation(int R, const double* arrival, const double* attn, int L, int wiring, double ffn,
             int min_batch, double max_wait)
      : R_(R), L_(L), wiring_(wiring), ffn_(ffn), min_batch_(min_batch), max_wait_(max_wait),
        attn_(attn), swept_(R * L, 0), joined_(R * L, 0), sweep_start_(R * L, NAN),
        sweep_end_(R * L, NAN), depart_(R * L, NAN), ret_(R * L, NAN), finish_(R, NAN),
        waiting_(L), free_at_(L, -INFINITY) {
    for (int r = 0; r < R; ++r) start_sweep(r, 0, arrival[r]);
  }

  // false if the run did not end within its bound on instants (it always does: every instant
  // holds a sweep end, a return, or the wake-up of a pool that departs or frees at that instant).
  bool run() {
    int64_t budget = 8 * (int64_t)R_ * L_ + 16;
    while (!events_.empty()) {
      if (--budget < 0) return false;
      const double t = events_.begin()->first;
      // completions at t, to a fixed point (handlers may add events at t)
      while (!events_.empty() && events_.begin()->first == t) {
        std::vector<Event> now = std::move(events_.begin()->second);
        events_.erase(events_.begin());
        for (const Event& e : now) handle(e, t);
      }
      for (int l = 0; l < L_; ++l) try_depart(l, t);
      for (int l = 0; l < L_; ++l) {
        if (waiting_[l].empty()) continue;
        if (free_at_[l] > t)
          events_[free_at_[l]];
        else if (isfinite(max_wait_))
          events_[fmax(deadline(l), t)];
      }
    }
    return true;
  }

  void copy_out(double* finish, double* sweep_start, double* sweep_end, double* depart,
                double* ret) const {
    for (int r = 0; r < R_; ++r) finish[r] = finish_[r];
    for (int i = 0; i < R_ * L_; ++i) {
      if (sweep_start) sweep_start[i] = sweep_start_[i];
      if (sweep_end) sweep_end[i] = sweep_end_[i];
      if (depart) depart[i] = depart_[i];
      if (ret) ret[i] = ret_[i];
    }
  }

 private:
  int idx(int r, int l) const { return r * L_ + l; }

  // The instant at which pool l's oldest waiting request has waited max_wait (+inf: never).
  double deadline(int l) const { return waiting_[l].front().first + max_wait_; }

  void start_sweep(int r, int l, double t) {
    sweep_start_[idx(r, l)] = t;
    sweep_end_[idx(r, l)] = t + attn_[r];
    events_[t + attn_[r]].push_back(Event{0, r, l, {}});
  }

  void join(int r, int l, double t) {
    if (joined_[idx(r, l)]) return;
    joined_[idx(r, l)] = 1;
    waiting_[l].emplace_back(t, r);
  }

  void ready(int r, int l, double t) {  // Q-First: layer l's output exists at t?
    if (!swept_[idx(r, l)] || joined_[idx(r, l)]) return;
    if (l > 0 && isnan(ret_[idx(r, l - 1)])) return;
    join(r, l, t);
    if (l + 1 < L_) start_sweep(r, l + 1, t);
  }

  void handle(const Event& e, double t) {
    if (e.kind == 0) {
      swept_[idx(e.r, e.l)] = 1;
      if (wiring_ == QF_WIRING_QFIRST)
        ready(e.r, e.l, t);
      else
        join(e.r, e.l, t);
    } else if (e.kind == 1) {
      for (int r : e.members) {
        ret_[idx(r, e.l)] = t;
        if (e.l + 1 == L_)
          finish_[r] = t;
        else if (wiring_ == QF_WIRING_QFIRST)
          ready(r, e.l + 1, t);
        else
          start_sweep(r, e.l + 1, t);
      }
    }
  }

  void try_depart(int l, double t) {
    std::deque<std::pair<double, int>>& q = waiting_[l];
    if (q.empty() || free_at_[l] > t) return;
    if ((int)q.size() < min_batch_ && !(t >= deadline(l))) return;
    Event e{1, -1, l, {}};
    for (const auto& w : q) {
      e.members.push_back(w.second);
      depart_[idx(w.second, l)] = t;
    }
    q.clear();
    free_at_[l] = t + ffn_;
    events_[t + ffn_].push_back(std::move(e));
  }

  const int R_, L_, wiring_;
  const double ffn_;
  const int min_batch_;
  const double max_wait_;
  const double* attn_;
  std::vector<char> swept_, joined_;
  std::vector<double> sweep_start_, sweep_end_, depart_, ret_, finish_;
  std::vector<std::deque<std::pair<double, int>>> waiting_;
  std::vector<double> free_at_;
  std::map<double, std::vector<Event>> events_;
};

}  // namespace

namespace qf {

// Arguments are checked by qf_schedule_simulate (qfattn_api.hip).
int simulate_schedule(int R, const double* arrival, const double* attn_time, int L, int wiring,
                      double ffn_time, int min_batch, double max_wait, double* finish,
                      double* sweep_start, double* sweep_end, double* ffn_depart,
                      double* ffn_return) {
  try {
    Simulation sim(R, arrival, attn_time, L, wiring, ffn_time, min_batch, max_wait);
    if (!sim.run()) return QF_EINVAL;
    sim.copy_out(finish, sweep_start, sweep_end, ffn_depart, ffn_return);
  } catch (...) {
    return QF_EINVAL;
  }
  return QF_OK;
}

}  // namespace qf
