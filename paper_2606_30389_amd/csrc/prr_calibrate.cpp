// Online calibration of the EMA predictor (Section 4.2): the score-weighted hit rate of
// Eq. (4) for every candidate theta = (alpha, beta, gamma) of a grid, simulated over
// prefill score trajectories, and its argmax (Eq. (5)).  Host code: it runs on the CPU
// cores while the device finishes the prefill, one grid point per task.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <thread>
#include <vector>

#include "prr_launch.h"

namespace {

// Order-preserving float -> uint32 map of the selection keys (-0 == +0); the decision
// values are rounded to float32 first, as on the device.
inline uint32_t key_of(double v) {
  float f = (float)v;
  if (f == 0.0f) f = 0.0f;
  uint32_t u;
  memcpy(&u, &f, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Membership (0/1 by block index) of the k largest of the packed candidates (ties:
// lower index first); `cand` holds only the blocks that may be chosen.
void top_k(std::vector<uint64_t>& cand, int k, std::vector<uint8_t>& in) {
  std::fill(in.begin(), in.end(), 0);
  const int n = (int)cand.size();
  if (k <= 0 || n == 0) return;
  if (k < n) std::nth_element(cand.begin(), cand.begin() + (k - 1), cand.end(), std::greater<uint64_t>());
  for (int i = 0; i < std::min(k, n); ++i) in[~(uint32_t)cand[i] & 0xffffffffu] = 1;
}

inline uint64_t pack(uint32_t key, int index) { return ((uint64_t)key << 32) | (uint32_t)~(uint32_t)index; }

// Eq. (4) for one theta over B trajectories of T rows of N scores, averaged over B.  Block
// i exists from row born[i] on (Section 4.1: its state starts there as level = its score,
// trend = 0); A_phi ranks the blocks that exist at row phi, P_phi the predictions of the
// blocks that had a state before it.  Rows phi >= 1 (those with a prediction) are averaged.
double objective(const float* scores, int B, int T, int N, const int32_t* born, int k, int p,
                 const float theta[3]) {
  const double alpha = theta[0], beta = theta[1], gamma = theta[2];
  std::vector<double> level(N), trend(N);
  std::vector<uint8_t> has(N), inA(N), inP(N);
  std::vector<uint64_t> cand;
  cand.reserve(N);
  double sum_b = 0.0;
  for (int b = 0; b < B; ++b) {
    const float* traj = scores + (size_t)b * T * N;
    std::fill(has.begin(), has.end(), 0);
    double sum_t = 0.0;
    int rows = 0;
    for (int phi = 0; phi < T; ++phi) {
      const float* row = traj + (size_t)phi * N;
      if (phi >= 1) {
        cand.clear();
        for (int i = 0; i < N; ++i)
          if (has[i]) cand.push_back(pack(key_of(level[i] + gamma * trend[i]), i));  // Eq. (2)
        top_k(cand, p, inP);
        cand.clear();
        for (int i = 0; i < N; ++i)
          if (born[i] <= phi) cand.push_back(pack(key_of(row[i]), i));
        top_k(cand, k, inA);
        double hit = 0.0, all = 0.0;
        for (int i = 0; i < N; ++i) {
          if (inA[i]) {
            all += row[i];
            if (inP[i]) hit += row[i];
          }
        }
        sum_t += all != 0.0 ? hit / all : 0.0;
        ++rows;
        for (int i = 0; i < N; ++i) {  // Eq. (3): the trend reads the previous level
          if (!has[i]) continue;
          trend[i] = beta * (row[i] - level[i]) + (1.0 - beta) * trend[i];
          level[i] = alpha * row[i] + (1.0 - alpha) * level[i];
        }
      }
      for (int i = 0; i < N; ++i) {  // blocks that form at this row
        if (!has[i] && born[i] <= phi) {
          level[i] = row[i];
          trend[i] = 0.0;
          has[i] = 1;
        }
      }
    }
    sum_b += rows ? sum_t / rows : 0.0;
  }
  return sum_b / B;
}

}  // namespace

namespace prr {

// Arguments were validated by the C ABI (prr_calibrate).
void calibrate_grid(const float* scores, int n_traj, int n_rows, int n_blocks, const int32_t* form_row, int k_select,
                    int p_select, const float* grid, int n_grid, int n_threads, float* best_theta,
                    double* objective_out) {
  const int p = p_select > 0 ? p_select : k_select;
  std::vector<int32_t> born(n_blocks, 0);
  if (form_row) born.assign(form_row, form_row + n_blocks);
  std::vector<double> obj(n_grid, 0.0);
  unsigned hw = std::thread::hardware_concurrency();
  int nt = n_threads > 0 ? n_threads : (int)(hw ? hw : 1);
  nt = std::max(1, std::min(nt, n_grid));
  std::atomic<int> next(0);
  auto work = [&]() {
    for (int g = next++; g < n_grid; g = next++)
      obj[g] = objective(scores, n_traj, n_rows, n_blocks, born.data(), k_select, p, grid + 3 * g);
  };
  std::vector<std::thread> pool;
  for (int i = 1; i < nt; ++i) pool.emplace_back(work);
  work();
  for (auto& th : pool) th.join();
  int best = 0;
  for (int g = 1; g < n_grid; ++g)
    if (obj[g] > obj[best]) best = g;  // the first grid point on ties
  for (int i = 0; i < 3; ++i) best_theta[i] = grid[3 * best + i];
  if (objective_out)
    for (int g = 0; g < n_grid; ++g) objective_out[g] = obj[g];
}

}  // namespace prr
