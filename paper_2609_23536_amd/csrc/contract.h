// Host-side bookkeeping contract of one pipeline stage (plain C++, no HIP).
//
// Implements the checks and commits of the paper's contract: TapeKey /
// TapeRef with generation-checked slots (§3.1, Invariant 2), the effect token
// advanced by the state-mutating actions only (§3.2, Invariant 1), weight and
// cache versions with first-forward refresh (§3.3, Invariant 3), arena views
// with exactly-once writes (§3.4, §4.3), and Algorithm 1's
// check -> physical action -> commit order with the failure rules of §4.5.
// A check never mutates state; a commit never fails.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "../../include/qe.h"

namespace qe {

constexpr uint32_t kBitDI = 1u, kBitDW = 2u;

inline bool key_eq(const qe_tape_key &a, const qe_tape_key &b) {
  return a.epoch == b.epoch && a.stage == b.stage && a.microbatch == b.microbatch && a.unit == b.unit &&
         a.invocation == b.invocation;
}

struct SlotState {
  bool live = false;
  qe_tape_key key{};
  uint32_t generation = 0;
  uint32_t bits = 0;
  int64_t tokens = 0;
};

struct View {
  bool bound = false;
  uintptr_t buf = 0;
  int64_t buf_elems = 0, offset = 0, ld = 0;
  bool written = false;
  uintptr_t start() const { return buf + 4u * uintptr_t(offset); }
};

struct LayerBook {
  uint32_t stage = 0, unit = 0;
  int64_t n = 0, k = 0, max_tokens = 0;
  int64_t e_c = -1;
  int64_t refreshes = 0;
  std::vector<SlotState> slots;
  std::vector<View> views;  // one per microbatch
  int64_t span(int64_t ld) const { return (n - 1) * ld + k; }
};

class Contract {
 public:
  explicit Contract(int microbatches) : M_(microbatches) {}

  int microbatches() const { return M_; }
  int num_layers() const { return int(layers_.size()); }
  const LayerBook &layer(int i) const { return layers_[size_t(i)]; }
  int64_t e_w() const { return e_w_; }
  int64_t token() const { return token_; }
  bool arena_valid() const { return arena_valid_; }
  bool finalized() const { return finalized_; }
  int64_t arena_bytes() const;

  int add_layer(uint32_t stage, uint32_t unit, int64_t n, int64_t k, int64_t max_tokens);
  bool has_layer(uint32_t stage, uint32_t unit) const;

  // F
  qe_status check_fwd(int layer, const qe_tape_key &key, int64_t tokens, bool *refresh) const;
  qe_tape_ref commit_fwd(int layer, const qe_tape_key &key, int64_t tokens, bool refresh);
  // dI
  qe_status check_dgrad(int layer, const qe_tape_key &key, const qe_tape_ref &ref) const;
  void commit_dgrad(int layer, const qe_tape_ref &ref);
  // dW with placement
  qe_status check_wgrad(int layer, const qe_tape_key &key, const qe_tape_ref &ref, uintptr_t buf, int64_t offset,
                        int64_t ld, int mode) const;
  void commit_wgrad(int layer, const qe_tape_ref &ref);
  // dI immediately followed by dW
  qe_status check_bwd_full(int layer, const qe_tape_key &key, const qe_tape_ref &ref, uintptr_t buf, int64_t offset,
                           int64_t ld, int mode) const;
  void commit_bwd_full(int layer, const qe_tape_ref &ref);

  qe_status bind(int layer, int64_t microbatch, uintptr_t buf, int64_t buf_elems, int64_t offset, int64_t ld);
  qe_status finalize();
  qe_status optimizer_commit();
  void abort_epoch();
  qe_status rebuild();

  // checkpoint (§3.5, Invariant 4): quiescence check, and the restart rule
  // (persistent e_W, caches stale; tapes, generations and token kept local)
  qe_status checkpoint_check() const;
  qe_status restore(int64_t e_w);

  // fault injection: the n-th next physical action fails
  void inject_fault(int32_t n) { fail_countdown_ = n; }
  bool physical_fails();

 private:
  qe_status resolve(int layer, const qe_tape_key &key, const qe_tape_ref &ref) const;
  qe_status check_dest(int layer, uint32_t m, uintptr_t buf, int64_t offset, int64_t ld, int mode) const;
  void release_if_done(SlotState &s);

  int M_;
  std::vector<LayerBook> layers_;
  int64_t e_w_ = 0;
  int64_t token_ = 0;
  bool arena_valid_ = true;
  bool finalized_ = false;
  int32_t fail_countdown_ = 0;
};

}  // namespace qe
