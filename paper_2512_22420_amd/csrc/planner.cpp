// The Nightjar speculative-length planner (Sec. 5.2, Algorithm 1): per batch
// size, a timeline of blocks and bins; a bin explores with probability 1/b_B
// and otherwise exploits Eq. (exploitation_min); the arm is locked for the
// bin.  Host code only.  The readings behind the open points (gamma_{t-1},
// unplayed arms, C_switch interpolation, ties) are listed in
// include/nightjar_planner.h.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "../../include/nightjar.h"
#include "../../include/nightjar_planner.h"
#include "kernels.h"

namespace {

constexpr int kMaxGamma = 15;
constexpr int kMaxBatch = 1 << 16;

struct BatchState {
  int32_t block = 1;  // j_B
  int64_t H = 1;      // H_B = 2^(j_B - 1)
  int64_t bin = 1;    // b_B
  int64_t tau = 1;    // tau_B
  int32_t gamma = 0;  // arm locked for the current bin
  int32_t prev = -1;  // arm of this B's previous step (prev_per_batch), -1 before the first
  int64_t steps = 0, bins = 0, explore_bins = 0;
};

struct Arm {
  double sum = 0.0;
  int64_t n = 0;
};

// tau > sqrt(H) and b > sqrt(H), exactly, in integers
bool exceeds_sqrt(int64_t v, int64_t H) { return v > 0 && (double)v * (double)v > (double)H; }

}  // namespace

struct nj_planner {
  nj_planner_config cfg;
  std::vector<BatchState> bs;  // [B - 1]
  std::vector<Arm> arms;       // [(B - 1) * (Gamma_max + 1) + gamma]
  uint64_t rng;
  int32_t prev_global = -1;    // arm of the previous step (any B), -1 before the first
  std::vector<int32_t> lengths, batches;
  std::vector<double> cost;    // [len][batch]

  // splitmix64 (Steele, Lea and Flood, 2014): the planner's exploration stream
  uint64_t next_u64() {
    uint64_t z = (rng += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  double uniform() { return (double)(next_u64() >> 11) * 0x1.0p-53; }  // [0, 1)

  Arm& arm(int B, int g) { return arms[(size_t)(B - 1) * (cfg.max_gamma + 1) + g]; }
  const Arm& arm(int B, int g) const { return arms[(size_t)(B - 1) * (cfg.max_gamma + 1) + g]; }
  double mean(int B, int g) const {
    const Arm& a = arm(B, g);
    return a.n ? a.sum / (double)a.n : cfg.unplayed_latency;
  }

  double switch_cost(int delta, int B) const {
    if (cost.empty()) return 0.0;
    const int nl = (int)lengths.size(), nb = (int)batches.size();
    // position along one axis: cell index and weight of the upper point
    auto locate = [](const std::vector<double>& axis, double v, int& i, double& w) {
      const int n = (int)axis.size();
      if (n == 1 || v <= axis[0]) {
        i = 0;
        w = 0.0;
        return;
      }
      if (v >= axis[n - 1]) {
        i = n - 2;
        w = 1.0;
        return;
      }
      i = (int)(std::upper_bound(axis.begin(), axis.end(), v) - axis.begin()) - 1;
      w = (v - axis[i]) / (axis[i + 1] - axis[i]);
    };
    std::vector<double> la(lengths.begin(), lengths.end()), ba(nb);
    for (int j = 0; j < nb; ++j) ba[j] = log2((double)batches[j]);
    int i, j;
    double wl, wb;
    locate(la, (double)delta, i, wl);
    locate(ba, log2((double)std::max(B, 1)), j, wb);
    auto at = [&](int a, int b) { return cost[(size_t)std::min(a, nl - 1) * nb + std::min(b, nb - 1)]; };
    const double c0 = (1 - wb) * at(i, j) + wb * at(i, j + 1);
    const double c1 = (1 - wb) * at(i + 1, j) + wb * at(i + 1, j + 1);
    return (1 - wl) * c0 + wl * c1;
  }
};

extern "C" {

nj_planner* nightjar_planner_create(const nj_planner_config* cfg) {
  if (!cfg) {
    nj::set_last_error(NJ_EINVAL, "planner config is NULL");
    return nullptr;
  }
  if (cfg->max_batch < 1 || cfg->max_batch > kMaxBatch) {
    nj::set_last_error(NJ_EINVAL, "max_batch must be in [1, %d]", kMaxBatch);
    return nullptr;
  }
  if (cfg->max_gamma < 0 || cfg->max_gamma > kMaxGamma) {
    nj::set_last_error(NJ_EINVAL, "max_gamma must be in [0, %d]", kMaxGamma);
    return nullptr;
  }
  if (!(cfg->unplayed_latency >= 0.0) || (cfg->prev_per_batch != 0 && cfg->prev_per_batch != 1)) {
    nj::set_last_error(NJ_EINVAL, "unplayed_latency must be >= 0 and prev_per_batch 0 or 1");
    return nullptr;
  }
  nj_planner* p = new nj_planner;
  p->cfg = *cfg;
  p->bs.resize(cfg->max_batch);
  p->arms.resize((size_t)cfg->max_batch * (cfg->max_gamma + 1));
  p->rng = cfg->seed;
  return p;
}

void nightjar_planner_destroy(nj_planner* p) { delete p; }

int nightjar_planner_set_switch_cost(nj_planner* p, const int32_t* lengths, int32_t n_lengths,
                                     const int32_t* batches, int32_t n_batches, const double* seconds) {
  if (!p || !lengths || !batches || !seconds || n_lengths < 1 || n_batches < 1)
    return nj::set_last_error(NJ_EINVAL, "switch-cost table: NULL pointer or empty axis");
  for (int i = 0; i < n_lengths; ++i)
    if (lengths[i] < 0 || (i && lengths[i] <= lengths[i - 1]))
      return nj::set_last_error(NJ_EINVAL, "switch-cost lengths must be >= 0 and strictly increasing");
  for (int j = 0; j < n_batches; ++j)
    if (batches[j] < 1 || (j && batches[j] <= batches[j - 1]))
      return nj::set_last_error(NJ_EINVAL, "switch-cost batch sizes must be >= 1 and strictly increasing");
  for (int i = 0; i < n_lengths * n_batches; ++i)
    if (!(seconds[i] >= 0.0) || !isfinite(seconds[i]))
      return nj::set_last_error(NJ_EINVAL, "switch costs must be finite and >= 0");
  p->lengths.assign(lengths, lengths + n_lengths);
  p->batches.assign(batches, batches + n_batches);
  p->cost.assign(seconds, seconds + (size_t)n_lengths * n_batches);
  return NJ_OK;
}

double nightjar_planner_switch_cost(const nj_planner* p, int32_t delta_max, int32_t B) {
  if (!p || delta_max < 0 || B < 1) {
    nj::set_last_error(NJ_EINVAL, "switch_cost: NULL planner, delta_max < 0 or B < 1");
    return -1.0;
  }
  return p->switch_cost(delta_max, B);
}

int nightjar_planner_select(nj_planner* p, int32_t B, int32_t delta_max, int32_t gamma_limit, int32_t* gamma) {
  if (!p || !gamma) return nj::set_last_error(NJ_EINVAL, "select: NULL planner or output");
  if (B < 1 || B > p->cfg.max_batch) return nj::set_last_error(NJ_EINVAL, "select: B outside [1, %d]", p->cfg.max_batch);
  if (delta_max < 0 || gamma_limit < 0) return nj::set_last_error(NJ_EINVAL, "select: delta_max and gamma_limit must be >= 0");
  const int limit = std::min(gamma_limit, p->cfg.max_gamma);
  BatchState& s = p->bs[B - 1];
  const int prev = p->cfg.prev_per_batch ? s.prev : p->prev_global;
  if (s.tau == 1) {  // bin start: explore with probability 1/b_B, else exploit
    ++s.bins;
    const double u = p->uniform();
    if (u < 1.0 / (double)s.bin) {
      s.gamma = std::min((int)(p->uniform() * (double)(limit + 1)), limit);
      ++s.explore_bins;
    } else {
      const double cs = prev == 0 ? p->switch_cost(delta_max, B) : 0.0;
      int best = 0;
      double best_v = INFINITY;
      for (int g = 0; g <= limit; ++g) {
        const double v = p->mean(B, g) + ((prev == 0 && g > 0) ? cs / (double)g : 0.0);
        if (v < best_v) {
          best_v = v;
          best = g;
        }
      }
      s.gamma = best;
    }
  }
  const int played = std::min(s.gamma, limit);
  *gamma = played;
  // the step is counted on B's timeline: advance the round, the bin, the block
  ++s.steps;
  ++s.tau;
  if (exceeds_sqrt(s.tau, s.H)) {
    ++s.bin;
    s.tau = 1;
    if (exceeds_sqrt(s.bin, s.H)) {
      ++s.block;
      s.H = (int64_t)1 << std::min(s.block - 1, 62);
      s.bin = 1;
    }
  }
  s.prev = played;
  p->prev_global = played;
  return NJ_OK;
}

int nightjar_planner_observe(nj_planner* p, int32_t B, int32_t gamma, double step_seconds, int32_t committed_tokens) {
  if (!p) return nj::set_last_error(NJ_EINVAL, "observe: NULL planner");
  if (B < 1 || B > p->cfg.max_batch || gamma < 0 || gamma > p->cfg.max_gamma)
    return nj::set_last_error(NJ_EINVAL, "observe: B or gamma out of range");
  if (!(step_seconds >= 0.0) || !isfinite(step_seconds) || committed_tokens < 1)
    return nj::set_last_error(NJ_EINVAL, "observe: step_seconds must be finite and >= 0, committed_tokens >= 1");
  Arm& a = p->arm(B, gamma);
  a.sum += step_seconds / (double)committed_tokens;
  ++a.n;
  return NJ_OK;
}

int nightjar_planner_bstate(const nj_planner* p, int32_t B, nj_planner_bstate* out) {
  if (!p || !out || B < 1 || B > p->cfg.max_batch) return nj::set_last_error(NJ_EINVAL, "bstate: bad arguments");
  const BatchState& s = p->bs[B - 1];
  *out = nj_planner_bstate{s.block, s.H, s.bin, s.tau, s.gamma, s.steps, s.bins, s.explore_bins};
  return NJ_OK;
}

int nightjar_planner_arm(const nj_planner* p, int32_t B, int32_t gamma, double* mean, int64_t* count) {
  if (!p || !mean || !count || B < 1 || B > p->cfg.max_batch || gamma < 0 || gamma > p->cfg.max_gamma)
    return nj::set_last_error(NJ_EINVAL, "arm: bad arguments");
  *mean = p->mean(B, gamma);
  *count = p->arm(B, gamma).n;
  return NJ_OK;
}

}  // extern "C"
