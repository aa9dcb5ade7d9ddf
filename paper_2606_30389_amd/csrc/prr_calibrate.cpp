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

// Membership (0/1 by block index) of the k largest of the candidates (keys key[j] of
// blocks idx[j]; ties: lower index first): two 11-bit radix passes narrow the rank-k key
// to one bin, whose few members are ordered exactly.
struct TopK {
  std::vector<uint32_t> hist;
  std::vector<uint64_t> tie;
  std::vector<int> sub;
  TopK() : hist(2048), tie(), sub() {}
};

inline uint64_t pack(uint32_t key, int index) { return ((uint64_t)key << 32) | (uint32_t)~(uint32_t)index; }

void top_k(const uint32_t* key, const int* idx, int n, int k, std::vector<uint8_t>& in, TopK& s) {
  std::fill(in.begin(), in.end(), 0);
  if (k <= 0 || n == 0) return;
  if (k >= n) {
    for (int j = 0; j < n; ++j) in[idx[j]] = 1;
    return;
  }
  // pass 1: bins of the top 11 bits; find the bin b1 holding rank k (from the top)
  std::fill(s.hist.begin(), s.hist.end(), 0u);
  for (int j = 0; j < n; ++j) ++s.hist[key[j] >> 21];
  int b1 = 2047, above = 0;
  while (above + (int)s.hist[b1] < k) above += s.hist[b1--];
  s.sub.clear();
  for (int j = 0; j < n; ++j) {
    const uint32_t b = key[j] >> 21;
    if ((int)b > b1) in[idx[j]] = 1;
    else if ((int)b == b1) s.sub.push_back(j);
  }
  // pass 2 within b1: the next 11 bits
  std::fill(s.hist.begin(), s.hist.end(), 0u);
  for (int j : s.sub) ++s.hist[(key[j] >> 10) & 2047u];
  int b2 = 2047;
  while (above + (int)s.hist[b2] < k) above += s.hist[b2--];
  s.tie.clear();
  for (int j : s.sub) {
    const int b = (int)((key[j] >> 10) & 2047u);
    if (b > b2) in[idx[j]] = 1;
    else if (b == b2) s.tie.push_back(pack(key[j], idx[j]));
  }
  // the members of the last bin: exact order by (key desc, index asc)
  const int need = k - above;
  if (need < (int)s.tie.size())
    std::nth_element(s.tie.begin(), s.tie.begin() + (need - 1), s.tie.end(), std::greater<uint64_t>());
  for (int j = 0; j < need; ++j) in[~(uint32_t)s.tie[j] & 0xffffffffu] = 1;
}

// A_phi of every row phi >= 1 of every trajectory (independent of theta): its blocks
// and their scores, and the denominator of Eq. (4).  Block i exists from row born[i] on.
struct RowSets {
  std::vector<std::vector<int>> idx;
  std::vector<std::vector<double>> w;
  std::vector<double> all;
};

RowSets row_sets(const float* scores, int B, int T, int N, const int32_t* born, int k, int nt) {
  RowSets R;
  R.idx.resize((size_t)B * T);
  R.w.resize((size_t)B * T);
  R.all.assign((size_t)B * T, 0.0);
  std::atomic<int> next(0);
  auto work = [&]() {
    std::vector<uint32_t> ck(N);
    std::vector<int> ci(N);
    std::vector<uint8_t> inA(N);
    TopK tk;
    for (int task = next++; task < B * T; task = next++) {
      const int b = task / T, phi = task % T;
      if (phi == 0) continue;
      const float* row = scores + ((size_t)b * T + phi) * N;
      int nc = 0;
      for (int i = 0; i < N; ++i) {
        if (born[i] <= phi) {
          ck[nc] = key_of(row[i]);
          ci[nc++] = i;
        }
      }
      top_k(ck.data(), ci.data(), nc, k, inA, tk);
      const size_t r = (size_t)b * T + phi;
      for (int i = 0; i < N; ++i) {
        if (inA[i]) {
          R.idx[r].push_back(i);
          R.w[r].push_back(row[i]);
          R.all[r] += row[i];
        }
      }
    }
  };
  std::vector<std::thread> pool;
  for (int i = 1; i < nt; ++i) pool.emplace_back(work);
  work();
  for (auto& th : pool) th.join();
  return R;
}

// Eq. (4) for one theta over B trajectories of T rows of N scores, averaged over B.  Block
// i exists from row born[i] on (Section 4.1: its state starts there as level = its score,
// trend = 0); P_phi ranks the predictions of the blocks that had a state before row phi,
// A_phi (precomputed) the blocks that exist at row phi.  Rows phi >= 1 (those with a
// prediction) are averaged.
double objective(const float* scores, int B, int T, int N, const int32_t* born, const RowSets& R, int p,
                 const float theta[3]) {
  const double alpha = theta[0], beta = theta[1], gamma = theta[2];
  std::vector<double> level(N), trend(N);
  std::vector<uint8_t> has(N), inP(N);
  std::vector<uint32_t> ck(N);
  std::vector<int> ci(N);
  TopK tk;
  double sum_b = 0.0;
  for (int b = 0; b < B; ++b) {
    const float* traj = scores + (size_t)b * T * N;
    std::fill(has.begin(), has.end(), 0);
    double sum_t = 0.0;
    int rows = 0;
    for (int phi = 0; phi < T; ++phi) {
      const float* row = traj + (size_t)phi * N;
      if (phi >= 1) {
        int nc = 0;
        for (int i = 0; i < N; ++i) {
          if (has[i]) {
            ck[nc] = key_of(level[i] + gamma * trend[i]);  // Eq. (2)
            ci[nc++] = i;
          }
        }
        top_k(ck.data(), ci.data(), nc, p, inP, tk);
        const size_t r = (size_t)b * T + phi;
        double hit = 0.0;
        const std::vector<int>& ia = R.idx[r];
        const std::vector<double>& wa = R.w[r];
        for (size_t j = 0; j < ia.size(); ++j)
          if (inP[ia[j]]) hit += wa[j];
        sum_t += R.all[r] != 0.0 ? hit / R.all[r] : 0.0;
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
  const int nt_all = std::max(1, n_threads > 0 ? n_threads : (int)(hw ? hw : 1));
  const RowSets R = row_sets(scores, n_traj, n_rows, n_blocks, born.data(), k_select,
                             std::min(nt_all, std::max(1, n_traj * n_rows)));
  const int nt = std::max(1, std::min(nt_all, n_grid));
  std::atomic<int> next(0);
  auto work = [&]() {
    for (int g = next++; g < n_grid; g = next++)
      obj[g] = objective(scores, n_traj, n_rows, n_blocks, born.data(), R, p, grid + 3 * g);
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
