// CacheScout's CPU control plane: the runtime state that decides which KV
// blocks to keep and which agent's anchor to prefetch (arXiv 2608.14624,
// Sec. 3 and the runtime workflow algorithm).
//
//   * Transition learner (Sec. 3.2): first-order counts C_ij of observed
//     agent transitions; Eq. (3) P_ij = (C_ij + eps) / sum_k (C_ik + eps);
//     Eq. (5) prediction = argmax_j P_ij.
//   * Survival scorer (Sec. 3.3): Eq. (7) keeps the edges with P(b|a) >= tau;
//     a breadth-first search from the current agent gives hop distances E[a];
//     Eq. (8) p~(a) = 1 - min(E[a], E_max) / E_max (0 when unreachable);
//     Eq. (9) Score(b) = (p~(a_b) + delta)(exp(-lambda age(b)) + delta)|b|,
//     the lowest score is evicted.
//   * Prefetch coordinator (Sec. 3.4): Eq. (2) predictability R over the
//     observed transitions, Eq. (11) gate R >= R_min, Eq. (10) target
//     a* = argmax_a P(a | a_t).
//
// Costs: a touch by the current agent is O(1); a dispatch (agent change)
// updates one counter and that row's entropy, O(A), and rebuilds the hop
// table, O(A^2) with the edges tested on the fly from the counts; survival
// and block scores read the cached hop table (the paper computes them once
// per scheduler step and refreshes the graph only on agent changes, Sec. 4);
// the predictability is O(A) from the cached row entropies and marginals.
#include "cachescout.h"
#include "error.h"

#include <math.h>

#include <new>
#include <unordered_map>
#include <vector>

// Edge tests, argmaxes and the gate compare fp64 values against thresholds;
// the file is built with -ffp-contract=off so each is evaluated as written.

struct cs_scout {
  int32_t num_agents;
  int32_t num_blocks;
  cs_scout_params prm;
  std::vector<uint32_t> counts;       // [A][A]
  std::vector<uint64_t> row_total;    // [A]
  std::vector<uint64_t> col_total;    // [A], successor marginal counts
  std::vector<double> row_entropy;    // [A], H(next | current = i), bits
  uint64_t transitions = 0;
  int32_t current = -1;
  std::vector<int32_t> hops;          // [A], -1 = unreachable
  std::vector<int32_t> queue;         // BFS scratch, [A]
  std::vector<int32_t> agent_of;      // [num_blocks], -1 = never touched
  std::vector<int64_t> last_access;   // [num_blocks]
  std::vector<int32_t> tokens;        // [num_blocks]
  std::vector<uint8_t> host_resident; // [num_blocks], contents also in the CPU tier
  std::unordered_map<uint64_t, int32_t> fingerprints;
};

namespace {

// Eq. (3); the denominator sum_k (C_ik + eps) is evaluated as
// (sum_k C_ik) + A * eps.
double prob_den(const cs_scout* s, int32_t i) {
  return (double)s->row_total[i] + (double)s->num_agents * s->prm.eps;
}

double prob(const cs_scout* s, int32_t i, int32_t j) {
  return ((double)s->counts[(size_t)i * s->num_agents + j] + s->prm.eps) / prob_den(s, i);
}

// Breadth-first hop distances from `src` over the edges with P >= tau.
void rebuild_hops(cs_scout* s, int32_t src) {
  const int32_t n = s->num_agents;
  for (int32_t a = 0; a < n; ++a) s->hops[a] = -1;
  s->hops[src] = 0;
  int32_t head = 0, tail = 0;
  s->queue[tail++] = src;
  while (head < tail) {
    const int32_t a = s->queue[head++];
    // Eq. (7): edge (a, b) iff P(b | a) >= tau
    const double den = prob_den(s, a);
    const uint32_t* row = &s->counts[(size_t)a * n];
    for (int32_t b = 0; b < n; ++b) {
      if (s->hops[b] < 0 && ((double)row[b] + s->prm.eps) / den >= s->prm.tau) {
        s->hops[b] = s->hops[a] + 1;
        s->queue[tail++] = b;
      }
    }
  }
}

double entropy_term(double p) { return p > 0.0 ? -p * log2(p) : 0.0; }

// Entropy of row i's empirical successor distribution; only the row whose
// count changed is recomputed, so Eq. (2) costs O(A) per dispatch and query.
void refresh_row_entropy(cs_scout* s, int32_t i) {
  const uint64_t ri = s->row_total[i];
  const uint32_t* row = &s->counts[(size_t)i * s->num_agents];
  double h = 0.0;
  for (int32_t j = 0; j < s->num_agents; ++j) h += entropy_term((double)row[j] / (double)ri);
  s->row_entropy[i] = h;
}

}  // namespace

// the C ABI is the only thing the library exports (built with -fvisibility=hidden)
#pragma GCC visibility push(default)
extern "C" {

void cs_scout_default_params(cs_scout_params* out) {
  if (!out) return;
  out->eps = 0.1;
  out->tau = 0.2;
  out->e_max = 4;
  out->lambda = 0.1;
  out->delta = 0.05;
  out->r_min = 0.3;
}

int cs_scout_create(int32_t num_agents, int32_t num_blocks, const cs_scout_params* params,
                    cs_scout** out) {
  if (!out) return cs::fail(CS_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  if (num_agents <= 0 || num_agents > 4096) return cs::fail(CS_ERR_INVALID_ARG, "num_agents %d outside [1, 4096]", num_agents);
  if (num_blocks < 0) return cs::fail(CS_ERR_INVALID_ARG, "num_blocks is negative");
  cs_scout_params prm;
  cs_scout_default_params(&prm);
  if (params) prm = *params;
  if (!(prm.eps > 0.0) || !(prm.tau >= 0.0 && prm.tau <= 1.0) || prm.e_max <= 0 ||
      !(prm.lambda >= 0.0) || !(prm.delta >= 0.0) || !isfinite(prm.r_min))
    return cs::fail(CS_ERR_INVALID_ARG, "parameters out of range (eps > 0, 0 <= tau <= 1, e_max > 0, lambda >= 0, delta >= 0)");
  cs_scout* s = new (std::nothrow) cs_scout();
  if (!s) return cs::fail(CS_ERR_INVALID_ARG, "out of host memory");
  s->num_agents = num_agents;
  s->num_blocks = num_blocks;
  s->prm = prm;
  s->counts.assign((size_t)num_agents * num_agents, 0);
  s->row_total.assign(num_agents, 0);
  s->col_total.assign(num_agents, 0);
  s->row_entropy.assign(num_agents, 0.0);
  s->hops.assign(num_agents, -1);
  s->queue.assign(num_agents, 0);
  s->agent_of.assign(num_blocks, -1);
  s->last_access.assign(num_blocks, 0);
  s->tokens.assign(num_blocks, 0);
  s->host_resident.assign(num_blocks, 0);
  *out = s;
  return cs::ok();
}

void cs_scout_destroy(cs_scout* s) { delete s; }

int32_t cs_scout_agent_id(cs_scout* s, uint64_t fingerprint) {
  if (!s) return -1;
  auto it = s->fingerprints.find(fingerprint);
  if (it != s->fingerprints.end()) return it->second;
  if ((int32_t)s->fingerprints.size() == s->num_agents) return -1;
  const int32_t id = (int32_t)s->fingerprints.size();
  s->fingerprints.emplace(fingerprint, id);
  return id;
}

int cs_scout_observe_touch(cs_scout* s, int32_t block, int32_t agent, int32_t tokens, int64_t now) {
  if (!s) return cs::fail(CS_ERR_INVALID_ARG, "null control-plane handle");
  if (tokens < 0) return cs::fail(CS_ERR_INVALID_ARG, "tokens %d is negative", tokens);
  if (block < 0 || block >= s->num_blocks) return cs::fail(CS_ERR_INVALID_ARG, "block %d outside [0, %d)", block, s->num_blocks);
  if (agent < 0 || agent >= s->num_agents) return cs::fail(CS_ERR_INVALID_ARG, "agent %d outside [0, %d)", agent, s->num_agents);
  s->agent_of[block] = agent;
  s->last_access[block] = now;
  s->tokens[block] = tokens;
  if (agent != s->current) {  // a dispatch to another agent
    if (s->current >= 0) {
      s->counts[(size_t)s->current * s->num_agents + agent] += 1;
      s->row_total[s->current] += 1;
      s->col_total[agent] += 1;
      s->transitions += 1;
      refresh_row_entropy(s, s->current);
    }
    rebuild_hops(s, agent);
    s->current = agent;
  }
  return cs::ok();
}

int cs_scout_observe_touches(cs_scout* s, const int32_t* blocks, const int32_t* agents,
                             const int32_t* tokens, const int64_t* now, int32_t n) {
  if (!s) return cs::fail(CS_ERR_INVALID_ARG, "null control-plane handle");
  if (n < 0) return cs::fail(CS_ERR_INVALID_ARG, "n is negative");
  if (n > 0 && (!blocks || !agents || !tokens || !now))
    return cs::fail(CS_ERR_INVALID_ARG, "null touch array");
  for (int32_t i = 0; i < n; ++i) {  // validate everything before changing anything
    if (blocks[i] < 0 || blocks[i] >= s->num_blocks)
      return cs::fail(CS_ERR_INVALID_ARG, "blocks[%d] = %d outside [0, %d)", i, blocks[i], s->num_blocks);
    if (agents[i] < 0 || agents[i] >= s->num_agents)
      return cs::fail(CS_ERR_INVALID_ARG, "agents[%d] = %d outside [0, %d)", i, agents[i], s->num_agents);
    if (tokens[i] < 0) return cs::fail(CS_ERR_INVALID_ARG, "tokens[%d] = %d is negative", i, tokens[i]);
  }
  for (int32_t i = 0; i < n; ++i) cs_scout_observe_touch(s, blocks[i], agents[i], tokens[i], now[i]);
  return cs::ok();
}

int32_t cs_scout_current(const cs_scout* s) { return s ? s->current : -1; }

double cs_scout_transition_prob(const cs_scout* s, int32_t i, int32_t j) {
  if (!s || i < 0 || i >= s->num_agents || j < 0 || j >= s->num_agents) return NAN;
  return prob(s, i, j);
}

int32_t cs_scout_predict(const cs_scout* s) {
  if (!s || s->current < 0) return -1;
  int32_t best = 0;
  double best_p = prob(s, s->current, 0);
  for (int32_t j = 1; j < s->num_agents; ++j) {
    const double p = prob(s, s->current, j);
    if (p > best_p) {
      best_p = p;
      best = j;
    }
  }
  return best;
}

double cs_scout_survival(const cs_scout* s, int32_t agent) {
  if (!s || agent < 0 || agent >= s->num_agents) return NAN;
  if (s->current < 0) return 0.0;
  const int32_t e = s->hops[agent];
  if (e < 0) return 0.0;
  const int32_t em = s->prm.e_max;
  return 1.0 - (double)(e < em ? e : em) / (double)em;
}

double cs_scout_score_block(const cs_scout* s, int32_t block, int64_t now) {
  if (!s || block < 0 || block >= s->num_blocks) return NAN;
  const int32_t a = s->agent_of[block];
  const double ps = a < 0 ? 0.0 : cs_scout_survival(s, a);
  const double age = (double)(now - s->last_access[block]);
  return (ps + s->prm.delta) * (exp(-s->prm.lambda * age) + s->prm.delta) * (double)s->tokens[block];
}

int cs_scout_set_host_resident(cs_scout* s, int32_t block, int32_t resident) {
  if (!s) return cs::fail(CS_ERR_INVALID_ARG, "null control-plane handle");
  if (block < 0 || block >= s->num_blocks)
    return cs::fail(CS_ERR_INVALID_ARG, "block %d outside [0, %d)", block, s->num_blocks);
  s->host_resident[block] = resident != 0;
  return cs::ok();
}

int32_t cs_scout_select_victim(const cs_scout* s, const int32_t* candidates, int32_t n, int64_t now) {
  if (!s || !candidates || n <= 0) return -1;
  int32_t best = -1;
  double best_score = INFINITY;
  bool best_resident = false;
  for (int32_t i = 0; i < n; ++i) {
    const double sc = cs_scout_score_block(s, candidates[i], now);
    if (isnan(sc)) return -1;
    // lowest score first; among equal scores a block already in the CPU tier
    const bool resident = s->host_resident[candidates[i]] != 0;
    if (best < 0 || sc < best_score || (sc == best_score && resident && !best_resident)) {
      best_score = sc;
      best_resident = resident;
      best = candidates[i];
    }
  }
  return best;
}

int cs_scout_survival_all(const cs_scout* s, double* out) {
  if (!s || !out) return cs::fail(CS_ERR_INVALID_ARG, "null handle or output");
  for (int32_t a = 0; a < s->num_agents; ++a) out[a] = cs_scout_survival(s, a);
  return cs::ok();
}

double cs_scout_predictability(const cs_scout* s) {
  if (!s) return NAN;
  if (s->transitions == 0) return 0.0;
  const int32_t n = s->num_agents;
  const double total = (double)s->transitions;
  double h_next = 0.0, h_cond = 0.0;
  for (int32_t j = 0; j < n; ++j) h_next += entropy_term((double)s->col_total[j] / total);
  for (int32_t i = 0; i < n; ++i) {
    const uint64_t ri = s->row_total[i];
    if (ri) h_cond += ((double)ri / total) * s->row_entropy[i];
  }
  if (h_next == 0.0) return 1.0;
  return 1.0 - h_cond / h_next;
}

int32_t cs_scout_between_step(const cs_scout* s) {
  if (!s || s->current < 0 || cs_scout_predictability(s) < s->prm.r_min) return -1;
  return cs_scout_predict(s);
}

int64_t cs_scout_state_bytes(const cs_scout* s) {
  if (!s) return -1;
  // transition counts, row and column totals, row entropies, hop table, block-to-agent map,
  // last-access, token and CPU-residency tables
  return (int64_t)s->counts.size() * sizeof(uint32_t) +
         (int64_t)s->row_total.size() * sizeof(uint64_t) +
         (int64_t)s->col_total.size() * sizeof(uint64_t) +
         (int64_t)s->row_entropy.size() * sizeof(double) +
         (int64_t)s->hops.size() * sizeof(int32_t) +
         (int64_t)s->num_blocks *
             (sizeof(int32_t) + sizeof(int64_t) + sizeof(int32_t) + sizeof(uint8_t));
}

}  // extern "C"
#pragma GCC visibility pop
