// The thief scheduler (section 4.2, Algorithm 1) with PickConfigs
// (Algorithm 2) and EstimateAccuracy.  Host code only.
//
// Models (the paper fixes the algorithms' steps, not these):
//  - an inference configuration needs a GPU share `cost` to keep up with its
//    live stream and reaches accuracy model_acc * factor; on a smaller share
//    it analyses only share / cost of the frames;
//  - PickConfigs takes, among the configurations that keep up on the
//    stream's inference share and whose accuracy acc_now * factor is at least
//    a_min, the most accurate (else the cheapest), then the retraining
//    configuration -- or none -- with the best window accuracy;
//  - EstimateAccuracy: retraining on share R lasts gpu_seconds / R (skipped
//    if longer than the window); the old model serves until it finishes, the
//    new one for the rest of the window;
//  - the fair start splits the quanta evenly over the jobs (the first jobs
//    take the remainder); a steal is kept only if it strictly improves.
#include <algorithm>
#include <cstddef>

#include "curve.hpp"

namespace ekya {

namespace {

double infer_acc(double model_acc, const SchedInfer& c, double share) {
  const double keep = share >= c.cost ? 1.0 : share / c.cost;
  return model_acc * c.factor * keep;
}

// Window accuracy; false if the retraining does not finish in the window.
bool estimate(const SchedVideo& v, const SchedTrain* t, const SchedInfer& ic, double ishare,
              double tshare, double T, double* acc) {
  if (!t) {
    *acc = infer_acc(v.acc_now, ic, ishare);
    return true;
  }
  if (tshare <= 0.0) return false;
  const double d = t->gpu_seconds / tshare;
  if (d > T) return false;
  *acc = (d * infer_acc(v.acc_now, ic, ishare) + (T - d) * infer_acc(t->acc_after, ic, ishare)) / T;
  return true;
}

double pick_configs(const std::vector<SchedVideo>& videos, const std::vector<int>& q, double delta,
                    double T, double a_min, SchedResult* r) {
  double sum = 0.0;
  r->infer_choice.assign(videos.size(), 0);
  r->train_choice.assign(videos.size(), -1);
  r->video_accuracy.assign(videos.size(), 0.0);
  for (size_t vi = 0; vi < videos.size(); ++vi) {
    const SchedVideo& v = videos[vi];
    const double ishare = q[2 * vi] * delta, tshare = q[2 * vi + 1] * delta;
    int bi = -1;
    for (size_t i = 0; i < v.infer.size(); ++i) {
      const SchedInfer& c = v.infer[i];
      if (c.cost <= ishare + 1e-12 && v.acc_now * c.factor >= a_min &&
          (bi < 0 || c.factor > v.infer[bi].factor))
        bi = (int)i;
    }
    if (bi < 0) {
      bi = 0;
      for (size_t i = 1; i < v.infer.size(); ++i)
        if (v.infer[i].cost < v.infer[bi].cost) bi = (int)i;
    }
    const SchedInfer& ic = v.infer[bi];
    double best = 0.0;
    estimate(v, nullptr, ic, ishare, tshare, T, &best);
    int bt = -1;
    for (size_t ti = 0; ti < v.train.size(); ++ti) {
      double a;
      if (estimate(v, &v.train[ti], ic, ishare, tshare, T, &a) && a > best) {
        best = a;
        bt = (int)ti;
      }
    }
    r->infer_choice[vi] = bi;
    r->train_choice[vi] = bt;
    r->video_accuracy[vi] = best;
    sum += best;
  }
  return sum / (double)videos.size();
}

}  // namespace

SchedResult thief_schedule(const std::vector<SchedVideo>& videos, int quanta, double delta,
                           double window_s, double a_min) {
  const int n_jobs = 2 * (int)videos.size();
  SchedResult best;
  best.quanta.assign(n_jobs, quanta / n_jobs);
  for (int j = 0; j < quanta % n_jobs; ++j) ++best.quanta[j];
  best.accuracy = pick_configs(videos, best.quanta, delta, window_s, a_min, &best);
  SchedResult trial;
  for (int thief = 0; thief < n_jobs; ++thief)
    for (int victim = 0; victim < n_jobs; ++victim) {
      if (thief == victim) continue;
      std::vector<int> temp = best.quanta;
      for (;;) {
        --temp[victim];
        ++temp[thief];
        if (temp[victim] < 0) break;
        const double acc = pick_configs(videos, temp, delta, window_s, a_min, &trial);
        if (acc > best.accuracy) {
          best = trial;
          best.quanta = temp;
          best.accuracy = acc;
        } else {
          break;
        }
      }
    }
  return best;
}

}  // namespace ekya
