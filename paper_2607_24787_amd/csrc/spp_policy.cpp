// Host-side availability policy (see spp_policy.h).
#include "spp_policy.h"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace spp {

SlotPolicy::SlotPolicy(int32_t S, int32_t n)
    : S_(S), n_(n), slot_expert_(S, kEmpty), slot_stamp_(S, 0), expert_slot_(n, kEmpty) {}

int32_t SlotPolicy::lowest_empty() const {
  for (int32_t j = 0; j < S_; ++j)
    if (slot_expert_[j] == kEmpty) return j;
  return kEmpty;
}

void SlotPolicy::put(int32_t slot, int32_t e) {
  const int32_t old = slot_expert_[slot];
  if (old != kEmpty) expert_slot_[old] = kEmpty;
  slot_expert_[slot] = e;
  expert_slot_[e] = slot;
}

bool SlotPolicy::set_resident(const int32_t* experts, int32_t count, std::string* err) {
  if (count < 0 || count > S_ || (count > 0 && !experts)) {
    *err = "resident count must be in [0, S]";
    return false;
  }
  std::vector<int32_t> table(S_, kEmpty);
  std::vector<int64_t> stamps(S_, 0);
  for (int32_t j = 0; j < count; ++j) table[j] = experts[j];
  return set_table(table.data(), stamps.data(), err);
}

bool SlotPolicy::set_table(const int32_t* experts, const int64_t* stamps, std::string* err) {
  std::vector<char> seen(n_, 0);
  for (int32_t j = 0; j < S_; ++j) {
    const int32_t e = experts[j];
    if (e == kEmpty) continue;
    if (e < 0 || e >= n_ || seen[e]) {
      *err = "slot table holds an out-of-range or duplicate expert";
      return false;
    }
    seen[e] = 1;
  }
  std::fill(expert_slot_.begin(), expert_slot_.end(), kEmpty);
  for (int32_t j = 0; j < S_; ++j) {
    slot_expert_[j] = experts[j];
    slot_stamp_[j] = stamps ? stamps[j] : 0;
    if (experts[j] != kEmpty) expert_slot_[experts[j]] = j;
  }
  return true;
}

int32_t SlotPolicy::distinct(const int32_t* needed, int32_t count) const {
  std::vector<char> seen(n_, 0);
  int32_t k = 0;
  for (int32_t i = 0; i < count; ++i) {
    const int32_t e = needed[i];
    if (e >= 0 && e < n_ && !seen[e]) {
      seen[e] = 1;
      ++k;
    }
  }
  return k;
}

bool SlotPolicy::on_demand(const int32_t* needed, int32_t count, int64_t tau, std::vector<Transfer>* loads,
                           std::vector<Round>* rounds, std::string* err) {
  std::vector<char> need(n_, 0);
  for (int32_t i = 0; i < count; ++i) {
    const int32_t e = needed[i];
    if (e < 0 || e >= n_) {
      *err = "needed expert id out of range";
      return false;
    }
    need[e] = 1;
  }
  loads->clear();
  rounds->clear();
  std::vector<int32_t> pending;
  for (int32_t e = 0; e < n_; ++e)
    if (need[e] && !available(e)) pending.push_back(e);
  std::vector<char> ran(n_, 0);
  size_t next = 0;
  for (int32_t round = 0;; ++round) {
    while (next < pending.size()) {
      int32_t v = lowest_empty();
      if (v == kEmpty) {
        for (int32_t j = 0; j < S_; ++j) {
          if (need[slot_expert_[j]]) continue;
          if (v == kEmpty || slot_stamp_[j] < slot_stamp_[v]) v = j;  // ties keep the lower slot
        }
      }
      if (v == kEmpty) {
        for (int32_t j = 0; j < S_; ++j)
          if (ran[slot_expert_[j]]) {
            v = j;
            break;
          }
      }
      if (v == kEmpty) break;
      const int32_t e = pending[next++];
      loads->push_back({e, v, slot_expert_[v], round});
      put(v, e);
    }
    Round run;
    for (int32_t e = 0; e < n_; ++e)
      if (need[e] && !ran[e] && available(e)) run.push_back({e, expert_slot_[e]});
    if (run.empty() && next < pending.size()) {
      *err = "on-demand rounds made no progress";  // cannot happen with S >= 1
      return false;
    }
    for (const auto& es : run) ran[es.first] = 1;
    rounds->push_back(std::move(run));
    if (next == pending.size()) break;
  }
  for (int32_t j = 0; j < S_; ++j)
    if (slot_expert_[j] != kEmpty && need[slot_expert_[j]]) slot_stamp_[j] = tau;
  return true;
}

void SlotPolicy::prefetch(const float* s, int32_t M_max, int64_t tau, std::vector<Transfer>* placed) {
  placed->clear();
  if (M_max <= 0) return;
  std::vector<int32_t> elig;
  elig.reserve(n_);
  for (int32_t e = 0; e < n_; ++e)
    if (!available(e) && !(std::isinf(s[e]) && s[e] < 0.f)) elig.push_back(e);
  // priority order: larger s first, lower index on equal s; NaN ranks last
  auto key_less = [s](int32_t a, int32_t b) {
    const float sa = s[a], sb = s[b];
    const bool na = std::isnan(sa), nb = std::isnan(sb);
    if (na != nb) return nb;
    if (!na && sa != sb) return sa > sb;
    return a < b;
  };
  const size_t m = std::min<size_t>(static_cast<size_t>(M_max), elig.size());
  std::partial_sort(elig.begin(), elig.begin() + m, elig.end(), key_less);
  for (size_t i = 0; i < m; ++i) {
    const int32_t e = elig[i];
    int32_t v = lowest_empty();
    if (v == kEmpty) {
      for (int32_t j = 0; j < S_; ++j) {
        if (slot_stamp_[j] >= tau) continue;
        if (v == kEmpty || slot_stamp_[j] < slot_stamp_[v]) v = j;
      }
    }
    if (v == kEmpty) break;
    placed->push_back({e, v, slot_expert_[v]});
    put(v, e);
    slot_stamp_[v] = tau;
  }
}

bool prefetch_budget(double window_us, double per_expert_cost_us, int32_t n, int32_t* out) {
  if (!std::isfinite(window_us) || !std::isfinite(per_expert_cost_us) || per_expert_cost_us <= 0.0 || n < 0)
    return false;
  if (window_us <= 0.0) {
    *out = 0;
    return true;
  }
  const double m = std::floor(window_us / per_expert_cost_us);
  *out = m >= static_cast<double>(n) ? n : static_cast<int32_t>(m);
  return true;
}

}  // namespace spp
