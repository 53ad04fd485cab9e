// Host-side bookkeeping contract (plain C++; see contract.h).
#include "contract.h"

namespace qe {

int Contract::add_layer(uint32_t stage, uint32_t unit, int64_t n, int64_t k, int64_t max_tokens) {
  LayerBook L;
  L.stage = stage;
  L.unit = unit;
  L.n = n;
  L.k = k;
  L.max_tokens = max_tokens;
  L.slots.assign(size_t(M_), SlotState{});
  L.views.assign(size_t(M_), View{});
  layers_.push_back(L);
  return int(layers_.size()) - 1;
}

bool Contract::has_layer(uint32_t stage, uint32_t unit) const {
  for (const auto &L : layers_)
    if (L.stage == stage && L.unit == unit) return true;
  return false;
}

int64_t Contract::arena_bytes() const {
  int64_t b = 0;
  for (const auto &L : layers_)
    for (const auto &v : L.views)
      if (v.bound) b += 4 * L.n * L.k;
  return b;
}

bool Contract::physical_fails() {
  if (fail_countdown_ > 0) {
    --fail_countdown_;
    if (fail_countdown_ == 0) return true;
  }
  return false;
}

// ---------------------------------------------------------------- F
qe_status Contract::check_fwd(int layer, const qe_tape_key &key, int64_t tokens, bool *refresh) const {
  *refresh = false;
  if (layer < 0 || layer >= num_layers()) return QE_ERR_INVALID_ARG;
  const LayerBook &L = layers_[size_t(layer)];
  if (key.stage != L.stage || key.unit != L.unit) return QE_ERR_KEY_MISMATCH;
  if (key.microbatch >= uint32_t(M_) || tokens < 0 || tokens > L.max_tokens) return QE_ERR_INVALID_ARG;
  if (int64_t(key.epoch) != e_w_) return QE_ERR_EPOCH;
  const SlotState &s = L.slots[key.microbatch];
  if (s.live) return key_eq(s.key, key) ? QE_ERR_KEY_LIVE : QE_ERR_POOL_FULL;
  const bool stale = L.e_c != e_w_;
  if (stale && key.microbatch != 0) return QE_ERR_STALE_CACHE;
  *refresh = stale;
  return QE_OK;
}

qe_tape_ref Contract::commit_fwd(int layer, const qe_tape_key &key, int64_t tokens, bool refresh) {
  LayerBook &L = layers_[size_t(layer)];
  SlotState &s = L.slots[key.microbatch];
  s.generation += 1;
  s.live = true;
  s.key = key;
  s.bits = 0;
  s.tokens = tokens;
  token_ += 1;
  if (refresh) {
    L.e_c = e_w_;
    L.refreshes += 1;
  }
  return qe_tape_ref{key.microbatch, s.generation};
}

// ---------------------------------------------------------------- shared checks
qe_status Contract::resolve(int layer, const qe_tape_key &key, const qe_tape_ref &ref) const {
  const LayerBook &L = layers_[size_t(layer)];
  if (ref.slot >= uint32_t(M_)) return QE_ERR_INVALID_ARG;
  const SlotState &s = L.slots[ref.slot];
  if (!s.live || s.generation != ref.generation) return QE_ERR_STALE_REF;
  if (!key_eq(s.key, key)) return QE_ERR_KEY_MISMATCH;
  if (int64_t(key.epoch) != e_w_) return QE_ERR_EPOCH;
  return QE_OK;
}

qe_status Contract::check_dest(int layer, uint32_t m, uintptr_t buf, int64_t offset, int64_t ld, int mode) const {
  const View &v = layers_[size_t(layer)].views[m];
  if (!v.bound || v.buf != buf || v.offset != offset || v.ld != ld) return QE_ERR_DEST_MISMATCH;
  if (v.written) return QE_ERR_DUP_WRITE;
  bool initialised = false;
  for (const auto &L : layers_)
    for (const auto &o : L.views)
      if (o.bound && o.written && o.start() == v.start() && o.ld == v.ld) initialised = true;
  if ((mode == QE_PLACE_INIT) == initialised) return QE_ERR_ORDER;
  return QE_OK;
}

void Contract::release_if_done(SlotState &s) {
  if (s.bits == (kBitDI | kBitDW)) {
    s.live = false;
    s.key = qe_tape_key{};
    s.tokens = 0;
  }
}

// ---------------------------------------------------------------- dI
qe_status Contract::check_dgrad(int layer, const qe_tape_key &key, const qe_tape_ref &ref) const {
  if (layer < 0 || layer >= num_layers()) return QE_ERR_INVALID_ARG;
  const qe_status st = resolve(layer, key, ref);
  if (st != QE_OK) return st;
  if (layers_[size_t(layer)].slots[ref.slot].bits & kBitDI) return QE_ERR_DUPLICATE_CONSUMER;
  return QE_OK;
}

void Contract::commit_dgrad(int layer, const qe_tape_ref &ref) {
  layers_[size_t(layer)].slots[ref.slot].bits |= kBitDI;
  token_ += 1;
}

// ---------------------------------------------------------------- dW
qe_status Contract::check_wgrad(int layer, const qe_tape_key &key, const qe_tape_ref &ref, uintptr_t buf,
                                int64_t offset, int64_t ld, int mode) const {
  if (layer < 0 || layer >= num_layers() || (mode != QE_PLACE_INIT && mode != QE_PLACE_ACCUM))
    return QE_ERR_INVALID_ARG;
  if (!arena_valid_) return QE_ERR_ARENA_INVALID;
  const qe_status st = resolve(layer, key, ref);
  if (st != QE_OK) return st;
  const uint32_t bits = layers_[size_t(layer)].slots[ref.slot].bits;
  if (!(bits & kBitDI)) return QE_ERR_ORDER;
  if (bits & kBitDW) return QE_ERR_DUPLICATE_CONSUMER;
  return check_dest(layer, ref.slot, buf, offset, ld, mode);
}

void Contract::commit_wgrad(int layer, const qe_tape_ref &ref) {
  LayerBook &L = layers_[size_t(layer)];
  SlotState &s = L.slots[ref.slot];
  s.bits |= kBitDW;
  L.views[ref.slot].written = true;
  release_if_done(s);
}

// ---------------------------------------------------------------- dI + dW
qe_status Contract::check_bwd_full(int layer, const qe_tape_key &key, const qe_tape_ref &ref, uintptr_t buf,
                                   int64_t offset, int64_t ld, int mode) const {
  if (layer < 0 || layer >= num_layers() || (mode != QE_PLACE_INIT && mode != QE_PLACE_ACCUM))
    return QE_ERR_INVALID_ARG;
  if (!arena_valid_) return QE_ERR_ARENA_INVALID;
  const qe_status st = resolve(layer, key, ref);
  if (st != QE_OK) return st;
  if (layers_[size_t(layer)].slots[ref.slot].bits & (kBitDI | kBitDW)) return QE_ERR_DUPLICATE_CONSUMER;
  return check_dest(layer, ref.slot, buf, offset, ld, mode);
}

void Contract::commit_bwd_full(int layer, const qe_tape_ref &ref) {
  LayerBook &L = layers_[size_t(layer)];
  SlotState &s = L.slots[ref.slot];
  s.bits |= kBitDI | kBitDW;
  token_ += 1;
  L.views[ref.slot].written = true;
  release_if_done(s);
}

// ---------------------------------------------------------------- arena
qe_status Contract::bind(int layer, int64_t microbatch, uintptr_t buf, int64_t buf_elems, int64_t offset,
                         int64_t ld) {
  if (layer < 0 || layer >= num_layers() || microbatch < 0 || microbatch >= M_) return QE_ERR_INVALID_ARG;
  LayerBook &L = layers_[size_t(layer)];
  if (buf == 0 || offset < 0 || ld < L.k || buf_elems < offset + L.span(ld)) return QE_ERR_INVALID_ARG;
  View &old = L.views[size_t(microbatch)];
  if (old.bound && old.written) return QE_ERR_DUP_WRITE;
  View nv;
  nv.bound = true;
  nv.buf = buf;
  nv.buf_elems = buf_elems;
  nv.offset = offset;
  nv.ld = ld;
  const uintptr_t lo = nv.start(), hi = lo + 4u * uintptr_t(L.span(ld));
  for (int l2 = 0; l2 < num_layers(); ++l2) {
    const LayerBook &L2 = layers_[size_t(l2)];
    for (int m2 = 0; m2 < M_; ++m2) {
      if (l2 == layer && m2 == microbatch) continue;
      const View &o = L2.views[size_t(m2)];
      if (!o.bound) continue;
      const uintptr_t olo = o.start(), ohi = olo + 4u * uintptr_t(L2.span(o.ld));
      if (lo < ohi && olo < hi) {
        const bool shared = l2 == layer && olo == lo && o.ld == ld;
        if (!shared) return QE_ERR_DEST_ALIAS;
      }
    }
  }
  old = nv;
  return QE_OK;
}

qe_status Contract::finalize() {
  if (!arena_valid_) return QE_ERR_ARENA_INVALID;
  for (const auto &L : layers_)
    for (const auto &v : L.views)
      if (v.bound && !v.written) return QE_ERR_INCOMPLETE;
  finalized_ = true;
  return QE_OK;
}

qe_status Contract::optimizer_commit() {
  bool any_bound = false;
  for (const auto &L : layers_) {
    for (const auto &s : L.slots)
      if (s.live) return QE_ERR_NOT_QUIESCENT;
    for (const auto &v : L.views) any_bound = any_bound || v.bound;
  }
  if (!arena_valid_) return QE_ERR_ARENA_INVALID;
  if (any_bound && !finalized_) return QE_ERR_INCOMPLETE;
  e_w_ += 1;
  for (auto &L : layers_)
    for (auto &v : L.views) v.written = false;
  finalized_ = false;
  return QE_OK;
}

void Contract::abort_epoch() {
  for (auto &L : layers_)
    for (auto &s : L.slots)
      if (s.live && int64_t(s.key.epoch) == e_w_) {
        s.live = false;
        s.key = qe_tape_key{};
        s.tokens = 0;
      }
  arena_valid_ = false;
  finalized_ = false;
}

qe_status Contract::rebuild() {
  arena_valid_ = true;
  for (auto &L : layers_)
    for (auto &v : L.views) v.written = false;
  finalized_ = false;
  return QE_OK;
}

qe_status Contract::checkpoint_check() const {
  for (const auto &L : layers_)
    for (const auto &s : L.slots)
      if (s.live) return QE_ERR_NOT_QUIESCENT;
  if (finalized_) return QE_ERR_NOT_QUIESCENT;
  for (const auto &L : layers_)
    for (const auto &v : L.views)
      if (v.written) return QE_ERR_NOT_QUIESCENT;
  if (!arena_valid_) return QE_ERR_ARENA_INVALID;
  return QE_OK;
}

qe_status Contract::restore(int64_t e_w) {
  const qe_status st = checkpoint_check();
  if (st != QE_OK) return st;
  e_w_ = e_w;
  for (auto &L : layers_) L.e_c = -1;
  return QE_OK;
}

}  // namespace qe
