// Host-side expert availability policy of one layer: the slot table that
// represents the available set, on-demand replacement, and the prefetch
// selection of Section "Window-Aware Prefetch Budgeting".  No HIP calls: the
// same object drives the device runtime and the host-only policy API.
#pragma once

#include <cstdint>
#include <string>
#include <utility>
#include <vector>

namespace spp {

constexpr int32_t kEmpty = -1;

struct Transfer {
  int32_t expert;
  int32_t slot;
  int32_t evicted;  // expert previously in the slot, or kEmpty
  int32_t round = 0;  // on-demand round the load belongs to
};

// (expert, slot) pairs that run in one round of an on-demand step.
using Round = std::vector<std::pair<int32_t, int32_t>>;

class SlotPolicy {
 public:
  SlotPolicy(int32_t S, int32_t n);

  int32_t S() const { return S_; }
  int32_t n() const { return n_; }
  int32_t slot_of(int32_t e) const { return expert_slot_[e]; }
  bool available(int32_t e) const { return expert_slot_[e] != kEmpty; }
  const std::vector<int32_t>& slot_experts() const { return slot_expert_; }
  const std::vector<int64_t>& slot_stamps() const { return slot_stamp_; }

  // Slots 0..count-1 take the listed experts with stamp 0; the rest are EMPTY.
  bool set_resident(const int32_t* experts, int32_t count, std::string* err);
  // Whole table (experts may be kEmpty); rejects duplicates / out-of-range ids.
  bool set_table(const int32_t* experts, const int64_t* stamps, std::string* err);

  // Load every distinct needed expert that is not available, in ascending
  // expert order, in rounds.  Victim = the lowest EMPTY slot, else the smallest
  // (stamp, slot index) among slots whose expert is not needed, else the
  // lowest-index slot whose expert already ran in an earlier round.  A round
  // loads while a victim exists, then runs every needed resident expert that
  // has not run yet (ascending expert); with at most S distinct needed experts
  // there is one round.  Then every slot holding a needed expert takes stamp
  // tau.  Fails (no change) if an id is out of range.
  bool on_demand(const int32_t* needed, int32_t count, int64_t tau, std::vector<Transfer>* loads,
                 std::vector<Round>* rounds, std::string* err);
  // Distinct experts among needed[0..count).
  int32_t distinct(const int32_t* needed, int32_t count) const;

  // P = the first M_max experts, not available and with s > -inf, in order
  // (s desc, index asc);
  // each placed in turn into the lowest EMPTY slot, else the smallest
  // (stamp, slot index) among slots stamped before tau; stops when no slot is
  // left.  Placed slots take stamp tau.
  void prefetch(const float* s, int32_t M_max, int64_t tau, std::vector<Transfer>* placed);

 private:
  int32_t lowest_empty() const;
  void put(int32_t slot, int32_t e);

  int32_t S_, n_;
  std::vector<int32_t> slot_expert_;
  std::vector<int64_t> slot_stamp_;
  std::vector<int32_t> expert_slot_;
};

// M_max = clamp(floor(W / c), 0, n); W <= 0 -> 0.  Returns false for a
// non-finite input, c <= 0 or n < 0.
bool prefetch_budget(double window_us, double per_expert_cost_us, int32_t n, int32_t* out);

}  // namespace spp
