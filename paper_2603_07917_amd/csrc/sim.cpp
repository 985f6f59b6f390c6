// Host-side discrete-event simulation of the request queue served in a given
// priority order: the replay behind sage_simulate. No GPU work happens here;
// the priority order comes from the library's index and rank kernels.
//
// Model (Sec. 3.2 cost, Sec. 3.3 preemptive Gittins scheduling refreshed at
// bucket boundaries, Sec. 4.1 Poisson arrivals, Sec. 4.4 bounded queue):
//   * a request needs C = O^2/2 + I*O cost units; after g generated tokens it
//     has received a(g) = g^2/2 + I*g;
//   * `servers` identical servers each run one request at a time and deliver
//     `rate` cost units per second;
//   * after every event instant (completions, then bucket boundaries, then
//     arrivals, all at that instant) the `servers` admitted requests with the
//     smallest keys run; a running request that drops out is preempted and
//     keeps what it received;
//   * at most queue_cap + servers requests are admitted and unfinished; later
//     arrivals wait outside, in arrival order;
//   * service accrues linearly within a run segment that starts at (t0, a0)
//     when a request starts, resumes or crosses a boundary (a0 = a(g) there).
//
// Keys are positions in `order`, a permutation of the entries e = k*R + r
// (request r after k boundaries). The keys are distinct, so every decision is
// an integer comparison: the floating-point decision is the ranking's.
// Positions >= `informed` hold entries without information (an index of +inf:
// no predicted mass above the service received); reaching such a level leaves
// the request's key unchanged.
#pragma clang fp contract(off)

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <functional>
#include <limits>
#include <queue>
#include <utility>
#include <vector>

namespace sage {

namespace {

struct Segment {
  int r;
  double t0, a0;     // start of the segment and the service received then
  double mark;       // service at the next boundary, or C if none is ahead
  double t_done;     // finish time if not interrupted
  double t_mark;     // next boundary time (+inf if none)
};

}  // namespace

// Returns 0 on success, -1 if the event loop stalls (cannot happen for inputs
// that pass sage_simulate's validation).
int simulate_queue(const double* arrival, const int32_t* prompt_len, const int32_t* output_len, int R,
                   const int32_t* order, int levels, int informed, int bucket, int servers,
                   double rate, int queue_cap, double* finish, int32_t* preemptions) {
  const double inf = std::numeric_limits<double>::infinity();
  std::vector<int32_t> key((size_t)levels * R);
  for (size_t i = 0; i < key.size(); ++i) key[order[i]] = (int32_t)i;

  std::vector<double> C(R), attained(R, 0.0);
  std::vector<int32_t> level(R, 0);
  std::vector<int32_t> cur(key.begin(), key.begin() + R);   // level-0 keys until refreshed
  for (int r = 0; r < R; ++r) {
    const double o = output_len[r], in = prompt_len[r];
    C[r] = o * o / 2.0 + in * o;
    if (preemptions) preemptions[r] = 0;
  }
  auto prio = [&](int r) { return cur[r]; };
  auto segment = [&](int r, double t) {
    Segment s;
    s.r = r;
    s.t0 = t;
    s.a0 = attained[r];
    const long long g_next = (long long)(level[r] + 1) * bucket;
    if (bucket > 0 && g_next < output_len[r]) {
      const double g = (double)g_next;
      s.mark = g * g / 2.0 + (double)prompt_len[r] * g;
      s.t_mark = t + (s.mark - s.a0) / rate;
    } else {
      s.mark = C[r];
      s.t_mark = inf;
    }
    s.t_done = t + (C[r] - s.a0) / rate;
    return s;
  };

  using Item = std::pair<int32_t, int32_t>;   // (key, request), smallest key on top
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> waiting;
  std::vector<Segment> run;
  run.reserve(servers);
  const long long cap = (long long)queue_cap + servers;
  long long pool = 0;
  int arrived = 0, admitted = 0, done = 0;

  while (done < R) {
    double t = arrived < R ? arrival[arrived] : inf;
    for (const Segment& s : run) t = std::min(t, std::min(s.t_done, s.t_mark));
    if (!(t < inf)) return -1;

    for (size_t i = 0; i < run.size();) {                  // completions
      if (run[i].t_done == t) {
        finish[run[i].r] = t;
        ++done;
        --pool;
        run[i] = run.back();
        run.pop_back();
      } else {
        ++i;
      }
    }
    for (Segment& s : run) {                                 // bucket boundaries
      if (s.t_mark == t) {
        ++level[s.r];
        attained[s.r] = s.mark;
        const int32_t k = key[(size_t)level[s.r] * R + s.r];
        if (k < informed) cur[s.r] = k;
        s = segment(s.r, t);
      }
    }
    while (arrived < R && arrival[arrived] == t) ++arrived;  // arrivals
    while (admitted < arrived && pool < cap) {
      waiting.push({prio(admitted), admitted});
      ++admitted;
      ++pool;
    }

    // Decision: fill idle servers, then swap the worst running request for
    // the best waiting one while that improves the running set.
    while (!waiting.empty()) {
      if ((int)run.size() < servers) {
        const int r = waiting.top().second;
        waiting.pop();
        run.push_back(segment(r, t));
        continue;
      }
      size_t worst = 0;
      for (size_t i = 1; i < run.size(); ++i)
        if (prio(run[i].r) > prio(run[worst].r)) worst = i;
      if (waiting.top().first >= prio(run[worst].r)) break;
      Segment& s = run[worst];
      attained[s.r] = std::min(s.a0 + (t - s.t0) * rate, s.mark);
      if (preemptions) ++preemptions[s.r];
      const int out = s.r;
      const int r = waiting.top().second;
      waiting.pop();
      waiting.push({prio(out), out});
      s = segment(r, t);
    }
  }
  return 0;
}

}  // namespace sage
