// Host-side computations of the scheduling layer: the micro-profiler's
// accuracy-curve fit (section 4.3) and the thief scheduler (section 4.2).
#pragma once

#include <vector>

namespace ekya {

// min || A x - b ||, x >= 0 (A row-major m x n); false on a singular
// least-squares subproblem.
bool nnls(const double* A, int m, int n, const double* b, double* x, double* rnorm);

// Held-out error after x passes over the window's data:
// 1 / (b0 x + b1) + b2, b0, b1, b2 >= 0.
struct Curve {
  double b0 = 0.0, b1 = 0.0, b2 = 0.0, rss = 0.0;
};
bool fit_accuracy_curve(const double* x, const double* acc, int n, Curve* out);
double curve_error(const Curve& c, double x);
double curve_accuracy(const Curve& c, double x);

struct SchedInfer {
  double cost, factor;
};
struct SchedTrain {
  double acc_after, gpu_seconds;
};
struct SchedVideo {
  double acc_now;
  std::vector<SchedInfer> infer;
  std::vector<SchedTrain> train;
};
struct SchedResult {
  std::vector<int> quanta;  // per job: infer v0, train v0, infer v1, ...
  std::vector<int> infer_choice, train_choice;
  std::vector<double> video_accuracy;
  double accuracy = 0.0;
};
SchedResult thief_schedule(const std::vector<SchedVideo>& videos, int quanta, double delta,
                           double window_s, double a_min);

}  // namespace ekya
