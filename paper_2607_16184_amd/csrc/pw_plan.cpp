// Runtime planner step (Sec. 3.2, Alg. 1), host code of libpagedweight.so.
//
// Damage model: Eq. 4 (global damage from the offline sensitivities), Eqs.
// 5-6 (prompt residual from routed-input features), Eq. 8 (bucket multiplier
// and damage floor); KV pressure as a byte target by Eq. 7; routing mass by
// Eq. 1 from the per-expert routing statistics.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <queue>
#include <string>
#include <vector>

#include "pw.h"
#include "pw_internal.hpp"

namespace {

constexpr int kBits[3] = {16, 8, 4};

int level_of(int bits) { return bits == 16 ? 0 : bits == 8 ? 1 : bits == 4 ? 2 : -1; }

struct Step {
  int unit, from, to;
};

struct StagePlan {
  bool valid = false;
  std::vector<Step> steps;           // in the order taken
  std::vector<int> from_bits;        // committed bitwidth of every unit the plan was built on
  uint64_t bytes = 0;
  double damage = 0.0;
};

}  // namespace

struct pw_planner {
  int E = 0, n = 0;
  std::vector<int> expert, type;
  std::vector<uint64_t> nbytes;      // [n][3]
  std::vector<double> sens;          // [n][3]
  pw_planner_config cfg{};
  // batch-level observation: KV-weighted sums of request masses and features
  std::vector<double> mass_w;        // [E]
  std::vector<double> phi_w;         // [E][2][3]
  double weight = 0.0;
  std::vector<StagePlan> queue;      // one candidate per stage (the plan queue)
  int selected = -1;
  pw_plan_summary last{};
};

namespace {

bool check_config(const pw_planner_config& c, std::string* err) {
  if (c.n_buckets < 1 || c.n_buckets > PW_PLAN_MAX_BUCKETS) { *err = "n_buckets out of range"; return false; }
  if (c.n_stages < 1 || c.n_stages > PW_PLAN_MAX_STAGES) { *err = "n_stages out of range"; return false; }
  for (int j = 0; j < c.n_buckets; ++j) {
    if (!(c.bucket_frac[j] >= 0.0) || !std::isfinite(c.bucket_frac[j])) { *err = "bad bucket fraction"; return false; }
    if (!(c.mult[j] >= 0.0) || !std::isfinite(c.mult[j])) { *err = "bad damage multiplier"; return false; }
    for (int s = 0; s < c.n_stages; ++s)
      if (level_of(c.floor_bits[s][j]) < 0) { *err = "bitwidth floors must be 16, 8 or 4"; return false; }
  }
  if (!(c.rho_min <= c.rho_max) || !std::isfinite(c.alpha) || !(c.eps >= 0.0)) {
    *err = "bad residual clip, strength or damage floor";
    return false;
  }
  return true;
}

// Experts sorted by mass (descending, ties to the lower index) into buckets.
std::vector<int> bucket_of(const pw_planner& p, const std::vector<double>& mass) {
  std::vector<int> order(p.E);
  for (int e = 0; e < p.E; ++e) order[e] = e;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return mass[a] > mass[b]; });
  std::vector<int> b(p.E, p.cfg.n_buckets - 1);
  double acc = 0.0;
  int start = 0;
  for (int j = 0; j < p.cfg.n_buckets; ++j) {
    acc += p.cfg.bucket_frac[j];
    const int end = j == p.cfg.n_buckets - 1 ? p.E : static_cast<int>(std::floor(p.E * acc + 0.5));
    for (int pos = start; pos < std::min(end, p.E); ++pos) b[order[pos]] = j;
    start = std::max(start, end);
  }
  return b;
}

// Eq. 8 for the one-level step of unit i from bitwidth level lv.
double step_damage(const pw_planner& p, int i, int lv, int bucket, const std::vector<double>& phi) {
  const pw_planner_config& c = p.cfg;
  const double g = std::max(p.sens[3 * i + lv + 1] - p.sens[3 * i + lv], 0.0);   // Eq. 4
  const int u = p.type[i];
  const double* f = &phi[(static_cast<size_t>(p.expert[i]) * 2 + u) * 3];
  double rho = 0.0;
  for (int k = 0; k < 3; ++k) rho += c.head_w[u][lv][k] * f[k];                  // Eq. 5
  rho += c.head_a[u][lv];
  rho = std::min(std::max(rho, c.rho_min), c.rho_max);
  const double eta = std::exp(c.alpha * c.head_c[u][lv] * rho);                  // Eq. 6
  return std::max(c.eps, c.mult[bucket] * g * eta);                              // Eq. 8
}

// ScoreActions + GreedySelect of one stage. Each unit offers at most one step
// at a time (its next level), so a heap keyed by (damage per byte, unit)
// takes the globally cheapest legal step each time.
StagePlan greedy(const pw_planner& p, const std::vector<int>& q, const std::vector<int>& bucket,
                 const std::vector<double>& phi, int stage, uint64_t D) {
  struct Cand {
    double ratio;
    int unit, lv;
    double dmg;
    uint64_t delta;
    bool operator>(const Cand& o) const { return ratio > o.ratio || (ratio == o.ratio && unit > o.unit); }
  };
  std::priority_queue<Cand, std::vector<Cand>, std::greater<Cand>> heap;
  auto offer = [&](int i, int lv) {
    if (lv < 0 || lv >= 2) return;
    const int b = bucket[p.expert[i]];
    if (kBits[lv + 1] < p.cfg.floor_bits[stage][b]) return;
    const uint64_t delta = p.nbytes[3 * i + lv] - p.nbytes[3 * i + lv + 1];
    if (delta == 0) return;
    const double d = step_damage(p, i, lv, b, phi);
    heap.push(Cand{d / static_cast<double>(delta), i, lv, d, delta});
  };
  for (int i = 0; i < p.n; ++i) offer(i, level_of(q[i]));
  StagePlan sp;
  sp.valid = true;
  sp.from_bits = q;
  while (sp.bytes < D && !heap.empty()) {
    const Cand c = heap.top();
    heap.pop();
    sp.steps.push_back(Step{c.unit, kBits[c.lv], kBits[c.lv + 1]});
    sp.bytes += c.delta;
    sp.damage += c.dmg;
    offer(c.unit, c.lv + 1);
  }
  return sp;
}

void collapse(const StagePlan& sp, std::vector<Step>* out) {
  out->clear();
  for (const Step& s : sp.steps) {
    auto it = std::find_if(out->begin(), out->end(), [&](const Step& o) { return o.unit == s.unit; });
    if (it == out->end()) out->push_back(s);
    else it->to = s.to;
  }
}

}  // namespace

extern "C" {

pw_status pw_planner_create(int n_experts, int n_units, const int* unit_expert, const int* unit_type,
                            const uint64_t* unit_bytes, const double* unit_sens, const pw_planner_config* cfg,
                            pw_planner** out) {
  if (!out) return pw::set_error(PW_EINVAL, "null output");
  *out = nullptr;
  if (n_experts < 1 || n_units < 0 || !cfg || (n_units > 0 && (!unit_expert || !unit_type || !unit_bytes || !unit_sens)))
    return pw::set_error(PW_EINVAL, "bad argument");
  std::string err;
  if (!check_config(*cfg, &err)) return pw::set_error(PW_EINVAL, err);
  for (int i = 0; i < n_units; ++i) {
    if (unit_expert[i] < 0 || unit_expert[i] >= n_experts) return pw::set_error(PW_EINVAL, "unit expert out of range");
    if (unit_type[i] != 0 && unit_type[i] != 1) return pw::set_error(PW_EINVAL, "unit type must be 0 or 1");
    if (unit_bytes[3 * i + 1] > unit_bytes[3 * i] || unit_bytes[3 * i + 2] > unit_bytes[3 * i + 1])
      return pw::set_error(PW_EINVAL, "unit sizes must not grow as the bitwidth falls");
    for (int j = 0; j < 3; ++j)
      if (!std::isfinite(unit_sens[3 * i + j])) return pw::set_error(PW_EINVAL, "non-finite sensitivity");
  }
  pw_planner* p = new pw_planner();
  p->E = n_experts;
  p->n = n_units;
  p->expert.assign(unit_expert, unit_expert + n_units);
  p->type.assign(unit_type, unit_type + n_units);
  p->nbytes.assign(unit_bytes, unit_bytes + 3 * static_cast<size_t>(n_units));
  p->sens.assign(unit_sens, unit_sens + 3 * static_cast<size_t>(n_units));
  p->cfg = *cfg;
  p->mass_w.assign(n_experts, 0.0);
  p->phi_w.assign(static_cast<size_t>(n_experts) * 6, 0.0);
  p->queue.resize(cfg->n_stages);
  p->last.stage = -1;
  *out = p;
  return PW_OK;
}

void pw_planner_destroy(pw_planner* p) { delete p; }

pw_status pw_planner_clear_requests(pw_planner* p) {
  if (!p) return pw::set_error(PW_EINVAL, "null planner");
  std::fill(p->mass_w.begin(), p->mass_w.end(), 0.0);
  std::fill(p->phi_w.begin(), p->phi_w.end(), 0.0);
  p->weight = 0.0;
  return PW_OK;
}

pw_status pw_planner_add_request(pw_planner* p, const double* sg, const double* sd, double kv_weight) {
  if (!p || !sg) return pw::set_error(PW_EINVAL, "bad argument");
  if (!(kv_weight > 0.0) || !std::isfinite(kv_weight)) return pw::set_error(PW_EINVAL, "KV weight must be positive");
  // Eq. 1 over the request's tokens, and its routed-input features
  double tot = 0.0;
  for (int e = 0; e < p->E; ++e) tot += sg[5 * e];
  for (int e = 0; e < p->E; ++e) {
    const double m = tot > 0.0 ? sg[5 * e] / tot : 0.0;
    p->mass_w[e] += kv_weight * m;
    for (int u = 0; u < 2; ++u) {
      const double* s = u == 0 ? sg + 5 * e : (sd ? sd + 5 * e : nullptr);
      if (!s || !(s[0] > 0.0)) continue;
      const double f[3] = {s[2] / s[0], std::sqrt(s[3] / s[0]), s[4]};
      for (int k = 0; k < 3; ++k) p->phi_w[(static_cast<size_t>(e) * 2 + u) * 3 + k] += kv_weight * f[k];
    }
  }
  p->weight += kv_weight;
  return PW_OK;
}

pw_status pw_planner_step(pw_planner* p, const int* q, int free_blocks, int free_threshold, uint64_t kv_block_bytes,
                          pw_plan_summary* out) {
  if (!p || (p->n > 0 && !q)) return pw::set_error(PW_EINVAL, "bad argument");
  for (int i = 0; i < p->n; ++i)
    if (q[i] != 0 && level_of(q[i]) < 0) return pw::set_error(PW_EINVAL, "unit bitwidths must be 16, 8, 4 or 0");
  // Eq. 7
  const int64_t blocks = std::max<int64_t>(0, static_cast<int64_t>(free_threshold) + 1 - free_blocks);
  const uint64_t D = static_cast<uint64_t>(blocks) * kv_block_bytes;
  // the batch-level table
  std::vector<double> mass(p->E, 0.0), phi(p->phi_w.size(), 0.0);
  if (p->weight > 0.0) {
    for (int e = 0; e < p->E; ++e) mass[e] = p->mass_w[e] / p->weight;
    for (size_t k = 0; k < phi.size(); ++k) phi[k] = p->phi_w[k] / p->weight;
  }
  const std::vector<int> bucket = bucket_of(*p, mass);
  const std::vector<int> qv(q, q + p->n);
  // one candidate per bitwidth-floor stage refreshes the queue
  for (int s = 0; s < p->cfg.n_stages; ++s) p->queue[s] = greedy(*p, qv, bucket, phi, s, D);
  pw_plan_summary r{};
  r.target = D;
  r.stage = -1;
  p->selected = -1;
  if (D > 0) {
    r.triggered = 1;
    int pick = -1;
    for (int s = 0; s < p->cfg.n_stages && pick < 0; ++s)
      if (p->queue[s].valid && p->queue[s].from_bits == qv && p->queue[s].bytes >= D) pick = s;
    if (pick < 0) {
      for (int s = 0; s < p->cfg.n_stages; ++s) {
        const StagePlan& c = p->queue[s];
        if (!c.valid || c.from_bits != qv) continue;
        if (pick < 0 || c.bytes > p->queue[pick].bytes ||
            (c.bytes == p->queue[pick].bytes && c.damage < p->queue[pick].damage))
          pick = s;
      }
    }
    if (pick >= 0) {
      const StagePlan& c = p->queue[pick];
      std::vector<Step> units;
      collapse(c, &units);
      r.stage = pick;
      r.bytes = c.bytes;
      r.damage = c.damage;
      r.n_steps = static_cast<int>(c.steps.size());
      r.n_units = static_cast<int>(units.size());
      p->selected = pick;
    }
  }
  p->last = r;
  if (out) *out = r;
  return PW_OK;
}

pw_status pw_planner_plan(const pw_planner* p, int stage, int steps, int max_n, int* unit, int* from_bits,
                          int* to_bits, uint64_t* bytes, int* n) {
  if (!p || !n || max_n < 0) return pw::set_error(PW_EINVAL, "bad argument");
  *n = 0;
  const int s = stage < 0 ? p->selected : stage;
  if (s < 0) return PW_OK;
  if (s >= p->cfg.n_stages) return pw::set_error(PW_EINVAL, "stage out of range");
  const StagePlan& c = p->queue[s];
  std::vector<Step> list;
  if (steps) list = c.steps;
  else collapse(c, &list);
  *n = static_cast<int>(list.size());
  for (int k = 0; k < std::min(max_n, *n); ++k) {
    const Step& st = list[k];
    if (unit) unit[k] = st.unit;
    if (from_bits) from_bits[k] = st.from;
    if (to_bits) to_bits[k] = st.to;
    if (bytes) bytes[k] = p->nbytes[3 * st.unit + level_of(st.from)] - p->nbytes[3 * st.unit + level_of(st.to)];
  }
  return PW_OK;
}

}  // extern "C"

namespace pw {

int planner_units(const pw_planner* p) { return p ? p->n : 0; }

}  // namespace pw
