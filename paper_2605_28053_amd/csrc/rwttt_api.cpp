// Host side of the RW-TTT READ/WRITE library: the owner table (versions,
// live/shadow slot bits, open candidates, tail lengths), the legal-group
// planner, and the C entry points declared in include/rwttt.h, dispatching to
// the fast-weight kernels (rwttt_kernels.hip) or the adapter kernels
// (rwttt_adapter.hip) by the context's backend.

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "rwttt.h"
#include "rwttt_kernels.h"

struct rwttt_ctx {
  rwttt_config cfg;
  std::vector<const void*> w0;       // [n_layers]
  std::vector<void*> slots;          // [n_owners * n_layers * 2]
  std::vector<uint8_t> live;         // [n_owners * n_layers]: which slot holds V(r)
  std::vector<uint8_t> written;      // [n_owners * n_layers]: shadow written in the open transition
  std::vector<uint64_t> version;     // [n_owners]: committed version V(r)
  std::vector<uint8_t> dirty;        // [n_owners]: a candidate is open
  std::vector<uint8_t> failed;       // [n_owners]: a WRITE of the open candidate failed
  std::vector<uint32_t> mark;        // [n_owners]: alias detection, epoch-stamped
  std::vector<void*> tail;           // [n_owners * n_layers] tail buffers, or empty
  std::vector<uint32_t> tail_len;    // [n_owners * n_layers] rows held
  uint32_t tail_rows = 0;
  uint32_t epoch = 0;
  uint32_t inject_failures = 0;
  int32_t last_hip = 0;

  size_t li(uint32_t owner, uint32_t layer) const { return size_t(owner) * cfg.n_layers + layer; }
  size_t io_bytes() const { return cfg.io_dtype == RWTTT_BF16 ? 2 : 4; }
  void* tail_row(uint32_t owner, uint32_t layer, uint32_t row) const {
    return static_cast<char*>(tail[li(owner, layer)]) + size_t(row) * cfg.d_ff * io_bytes();
  }
  // An update boundary closed (commit or rollback): the owner's tails empty.
  void clear_tail(uint32_t owner) {
    if (tail.empty()) return;
    for (uint32_t l = 0; l < cfg.n_layers; ++l) tail_len[li(owner, l)] = 0;
  }
  void* slot(uint32_t owner, uint32_t layer, int which) const {
    const int s = live[li(owner, layer)] ^ which;
    return slots[li(owner, layer) * 2 + s];
  }
  // Returns false if an owner id repeats or is out of range.
  bool distinct_owners(const uint32_t* owners, uint32_t n, rwttt_status* why) {
    if (++epoch == 0) {
      std::fill(mark.begin(), mark.end(), 0u);
      epoch = 1;
    }
    for (uint32_t i = 0; i < n; ++i) {
      const uint32_t r = owners[i];
      if (r >= cfg.n_owners) {
        *why = RWTTT_E_INVALID;
        return false;
      }
      if (mark[r] == epoch) {
        *why = RWTTT_E_OWNER_ALIAS;
        return false;
      }
      mark[r] = epoch;
    }
    return true;
  }
};

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool valid_dtype(int32_t d) { return d == RWTTT_F32 || d == RWTTT_BF16; }

rwttt_status check_shape(const rwttt_config* c) {
  if (!c) return RWTTT_E_INVALID;
  if (c->n_owners == 0 || c->n_layers == 0) return RWTTT_E_INVALID;
  if (c->d_ff < 8 || c->d_ff % 8 || c->d_model < 8 || c->d_model % 8) return RWTTT_E_INVALID;
  if (c->d_ff > (1u << 20) || c->d_model > (1u << 20)) return RWTTT_E_INVALID;
  if (!valid_dtype(c->io_dtype) || !valid_dtype(c->state_dtype)) return RWTTT_E_INVALID;
  if (c->max_group == 0 || c->max_group > RWTTT_MAX_GROUP) return RWTTT_E_INVALID;
  if (c->reserved != 0) return RWTTT_E_INVALID;
  if (c->backend == RWTTT_FAST_WEIGHT) {
    if (c->rank != 0) return RWTTT_E_INVALID;
  } else if (c->backend == RWTTT_DELTA_ADAPTER) {
    if (c->rank == 0 || c->rank > RWTTT_MAX_RANK) return RWTTT_E_INVALID;
  } else {
    return RWTTT_E_INVALID;
  }
  return RWTTT_OK;
}

bool is_adapter(const rwttt_config* c) { return c->backend == RWTTT_DELTA_ADAPTER; }

size_t slot_bytes_of(const rwttt_config* c) {
  const size_t s = c->state_dtype == RWTTT_BF16 ? 2 : 4;
  if (is_adapter(c)) return (size_t(c->d_ff) + c->d_model) * c->rank * s;
  return size_t(c->d_ff) * c->d_model * s;
}

size_t workspace_bytes_of(const rwttt_config* c) {
  if (is_adapter(c))
    return rwttt::adapter_geometry(int(c->d_ff), int(c->d_model), c->io_dtype == RWTTT_BF16,
                                   int(c->rank), int(c->n_owners))
        .total_bytes;
  return rwttt::read_geometry(int(c->d_ff), int(c->d_model), c->state_dtype == RWTTT_BF16,
                              int(c->n_owners))
      .total_bytes;
}

rwttt_status hip_fail(rwttt_ctx* ctx, hipError_t e) {
  ctx->last_hip = static_cast<int32_t>(e);
  return RWTTT_E_HIP;
}

}  // namespace

extern "C" {

rwttt_status rwttt_workspace_bytes(const rwttt_config* cfg, size_t* bytes) {
  const rwttt_status s = check_shape(cfg);
  if (s != RWTTT_OK) return s;
  if (!bytes) return RWTTT_E_INVALID;
  *bytes = workspace_bytes_of(cfg);
  return RWTTT_OK;
}

rwttt_status rwttt_slot_bytes(const rwttt_config* cfg, size_t* bytes) {
  const rwttt_status s = check_shape(cfg);
  if (s != RWTTT_OK) return s;
  if (!bytes) return RWTTT_E_INVALID;
  *bytes = slot_bytes_of(cfg);
  return RWTTT_OK;
}

rwttt_status rwttt_create(const rwttt_config* cfg, rwttt_ctx** out) {
  rwttt_status s = check_shape(cfg);
  if (s != RWTTT_OK) return s;
  if (!out || !cfg->w0 || !cfg->slots) return RWTTT_E_INVALID;
  const size_t n_slots = size_t(cfg->n_owners) * cfg->n_layers * 2;
  for (uint32_t l = 0; l < cfg->n_layers; ++l)
    if (!cfg->w0[l] || !aligned16(cfg->w0[l])) return RWTTT_E_INVALID;
  std::vector<void*> sorted(cfg->slots, cfg->slots + n_slots);
  for (void* p : sorted)
    if (!p || !aligned16(p)) return RWTTT_E_INVALID;
  std::sort(sorted.begin(), sorted.end());
  if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end()) return RWTTT_E_OWNER_ALIAS;
  if (cfg->workspace) {
    if ((reinterpret_cast<uintptr_t>(cfg->workspace) & 255u) != 0) return RWTTT_E_INVALID;
    if (cfg->workspace_bytes < workspace_bytes_of(cfg)) return RWTTT_E_CAPACITY;
  }

  rwttt_ctx* ctx = new (std::nothrow) rwttt_ctx;
  if (!ctx) return RWTTT_E_INVALID;
  ctx->cfg = *cfg;
  ctx->cfg.w0 = nullptr;
  ctx->cfg.slots = nullptr;
  ctx->w0.assign(cfg->w0, cfg->w0 + cfg->n_layers);
  ctx->slots.assign(cfg->slots, cfg->slots + n_slots);
  const size_t nl = size_t(cfg->n_owners) * cfg->n_layers;
  ctx->live.assign(nl, 0);
  ctx->written.assign(nl, 0);
  ctx->version.assign(cfg->n_owners, 0);
  ctx->dirty.assign(cfg->n_owners, 0);
  ctx->failed.assign(cfg->n_owners, 0);
  ctx->mark.assign(cfg->n_owners, 0);
  *out = ctx;
  return RWTTT_OK;
}

rwttt_status rwttt_destroy(rwttt_ctx* ctx) {
  if (!ctx) return RWTTT_E_INVALID;
  delete ctx;
  return RWTTT_OK;
}

rwttt_status rwttt_plan(const rwttt_ctx* ctx, const rwttt_event* ev, uint32_t n_ev, uint64_t step,
                        uint32_t target_b, uint32_t wait_budget, rwttt_group* groups,
                        uint32_t groups_cap, uint32_t* n_groups, uint32_t* owner_map, uint32_t map_cap,
                        uint32_t* n_mapped, uint32_t* deferred, uint32_t deferred_cap,
                        uint32_t* n_deferred, int32_t* ev_status) {
  if (!ctx || !n_groups || !n_mapped || !n_deferred) return RWTTT_E_INVALID;
  if (n_ev && (!ev || !ev_status)) return RWTTT_E_INVALID;
  if ((groups_cap && !groups) || (map_cap && !owner_map) || (deferred_cap && !deferred))
    return RWTTT_E_INVALID;
  *n_groups = *n_mapped = *n_deferred = 0;
  const uint32_t n_owners = ctx->cfg.n_owners;

  // One request exposes one next transition: an owner named twice is an alias.
  std::vector<uint8_t> seen(n_owners, 0);
  for (uint32_t i = 0; i < n_ev; ++i) {
    const uint32_t r = ev[i].owner;
    if (r < n_owners) {
      if (seen[r]) {
        for (uint32_t j = 0; j < n_ev; ++j) ev_status[j] = RWTTT_E_OWNER_ALIAS;
        return RWTTT_E_OWNER_ALIAS;
      }
      seen[r] = 1;
    }
  }

  std::vector<uint32_t> valid;
  valid.reserve(n_ev);
  for (uint32_t i = 0; i < n_ev; ++i) {
    const rwttt_event& e = ev[i];
    if ((e.effect != RWTTT_READ && e.effect != RWTTT_WRITE) || e.owner >= n_owners ||
        e.ready_step > step || e.reserved != 0) {
      ev_status[i] = RWTTT_E_INVALID;
    } else if (ctx->dirty[e.owner]) {
      ev_status[i] = RWTTT_E_DIRTY;
    } else if (e.expected_version != ctx->version[e.owner]) {
      ev_status[i] = RWTTT_E_STALE_VERSION;
    } else {
      ev_status[i] = RWTTT_OK;
      valid.push_back(i);
    }
  }

  // kappa = (rho, tau, sigma, pi), then (ready_step, owner) inside a key.
  auto key_less = [&](uint32_t a, uint32_t b) {
    const rwttt_event& x = ev[a];
    const rwttt_event& y = ev[b];
    if (x.effect != y.effect) return x.effect < y.effect;
    if (x.backend_type != y.backend_type) return x.backend_type < y.backend_type;
    if (x.shape_class != y.shape_class) return x.shape_class < y.shape_class;
    if (x.placement != y.placement) return x.placement < y.placement;
    if (x.ready_step != y.ready_step) return x.ready_step < y.ready_step;
    return x.owner < y.owner;
  };
  auto same_key = [&](uint32_t a, uint32_t b) {
    const rwttt_event& x = ev[a];
    const rwttt_event& y = ev[b];
    return x.effect == y.effect && x.backend_type == y.backend_type &&
           x.shape_class == y.shape_class && x.placement == y.placement;
  };
  std::sort(valid.begin(), valid.end(), key_less);

  uint32_t ng = 0, nm = 0, nd = 0;
  auto emit = [&](size_t lo, size_t hi) {
    if (ng < groups_cap) {
      const rwttt_event& e = ev[valid[lo]];
      rwttt_group& g = groups[ng];
      g.effect = e.effect;
      g.backend_type = e.backend_type;
      g.shape_class = e.shape_class;
      g.placement = e.placement;
      g.first = nm;
      g.count = uint32_t(hi - lo);
    }
    for (size_t i = lo; i < hi; ++i) {
      if (nm < map_cap) owner_map[nm] = ev[valid[i]].owner;
      ++nm;
    }
    ++ng;
  };

  size_t s = 0;
  while (s < valid.size()) {
    size_t e = s + 1;
    while (e < valid.size() && same_key(valid[s], valid[e])) ++e;
    size_t rest = s;
    if (target_b > 0) {
      const size_t full = (e - s) / target_b;
      for (size_t f = 0; f < full; ++f) emit(s + f * target_b, s + (f + 1) * target_b);
      rest = s + full * target_b;
    }
    if (rest < e) {
      // Members are sorted by ready step, so the oldest of the rest is first.
      const uint64_t oldest = ev[valid[rest]].ready_step;
      if (wait_budget == 0 || step - oldest >= wait_budget) {
        emit(rest, e);
      } else {
        for (size_t i = rest; i < e; ++i) {
          ev_status[valid[i]] = RWTTT_DEFERRED;
          if (nd < deferred_cap) deferred[nd] = valid[i];
          ++nd;
        }
      }
    }
    s = e;
  }
  *n_groups = ng;
  *n_mapped = nm;
  *n_deferred = nd;
  if (ng > groups_cap || nm > map_cap || nd > deferred_cap) return RWTTT_E_CAPACITY;
  return RWTTT_OK;
}

namespace {

// Defence in depth beside the planner (Section 3, eq. compatibility): every
// member must still be at the version the caller planned it at.
bool versions_match(const rwttt_ctx* ctx, const uint32_t* owners, const uint64_t* expected, uint32_t n) {
  if (!expected) return true;
  for (uint32_t b = 0; b < n; ++b)
    if (expected[b] != ctx->version[owners[b]]) return false;
  return true;
}

rwttt_status read_impl(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                       const uint64_t* expected, uint32_t layer, const void* x, void* y, void* stream,
                       bool append) {
  if (!ctx || !group) return RWTTT_E_INVALID;
  if (group->effect != RWTTT_READ && group->effect != RWTTT_WRITE) return RWTTT_E_INVALID;
  const uint32_t n = group->count;
  if (n == 0) return RWTTT_OK;
  if (!owner_map || !x || !y || layer >= ctx->cfg.n_layers) return RWTTT_E_INVALID;
  if (n > ctx->cfg.max_group) return RWTTT_E_CAPACITY;
  const uint32_t* owners = owner_map + group->first;
  rwttt_status why = RWTTT_OK;
  if (!ctx->distinct_owners(owners, n, &why)) return why;
  if (!versions_match(ctx, owners, expected ? expected + group->first : nullptr, n))
    return RWTTT_E_STALE_VERSION;
  if (!ctx->cfg.workspace) return RWTTT_E_INVALID;
  if (append) {
    if (ctx->tail.empty() || !aligned16(x)) return RWTTT_E_INVALID;
    for (uint32_t b = 0; b < n; ++b)
      if (ctx->tail_len[ctx->li(owners[b], layer)] >= ctx->tail_rows) return RWTTT_E_CAPACITY;
  }

  if (is_adapter(&ctx->cfg)) {
    rwttt::AdapterReadLaunch A;
    A.io_bf16 = ctx->cfg.io_dtype == RWTTT_BF16;
    A.state_bf16 = ctx->cfg.state_dtype == RWTTT_BF16;
    A.d_ff = int(ctx->cfg.d_ff);
    A.d_model = int(ctx->cfg.d_model);
    A.rank = int(ctx->cfg.rank);
    A.count = int(n);
    A.n_owners = int(ctx->cfg.n_owners);
    A.x = x;
    A.y = y;
    A.w0 = ctx->w0[layer];
    A.workspace = ctx->cfg.workspace;
    for (uint32_t b = 0; b < n; ++b) {
      const uint32_t r = owners[b];
      A.state[b] = ctx->slot(r, layer, 0);
      A.row[b] = r;
      A.tail[b] = append ? ctx->tail_row(r, layer, ctx->tail_len[ctx->li(r, layer)]) : nullptr;
    }
    const hipError_t e = rwttt::launch_adapter_read(A, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(ctx, e);
    if (append)
      for (uint32_t b = 0; b < n; ++b) ++ctx->tail_len[ctx->li(owners[b], layer)];
    return RWTTT_OK;
  }

  rwttt::ReadLaunch L;
  L.io_bf16 = ctx->cfg.io_dtype == RWTTT_BF16;
  L.state_bf16 = ctx->cfg.state_dtype == RWTTT_BF16;
  L.d_ff = int(ctx->cfg.d_ff);
  L.d_model = int(ctx->cfg.d_model);
  L.count = int(n);
  L.n_owners = int(ctx->cfg.n_owners);
  L.x = x;
  L.y = y;
  L.w0 = ctx->w0[layer];
  L.workspace = ctx->cfg.workspace;
  for (uint32_t b = 0; b < n; ++b) {
    const uint32_t r = owners[b];
    L.dw[b] = ctx->slot(r, layer, 0);
    L.row[b] = r;
    L.tail[b] = append ? ctx->tail_row(r, layer, ctx->tail_len[ctx->li(r, layer)]) : nullptr;
  }
  const hipError_t e = rwttt::launch_read(L, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(ctx, e);
  if (append)
    for (uint32_t b = 0; b < n; ++b) ++ctx->tail_len[ctx->li(owners[b], layer)];
  return RWTTT_OK;
}

}  // namespace

rwttt_status rwttt_read(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                        const uint64_t* expected, uint32_t layer, const void* x, void* y, void* stream) {
  return read_impl(ctx, group, owner_map, expected, layer, x, y, stream, false);
}

rwttt_status rwttt_read_append(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                               const uint64_t* expected, uint32_t layer, const void* x, void* y,
                               void* stream) {
  return read_impl(ctx, group, owner_map, expected, layer, x, y, stream, true);
}

rwttt_status rwttt_read_noalloc(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                                const uint64_t* expected, uint32_t layer, const void* x, void* y,
                                void* stream) {
  if (!ctx || !group) return RWTTT_E_INVALID;
  if (group->effect != RWTTT_READ && group->effect != RWTTT_WRITE) return RWTTT_E_INVALID;
  if (is_adapter(&ctx->cfg)) return RWTTT_E_INVALID;
  const uint32_t n = group->count;
  if (n == 0) return RWTTT_OK;
  if (!owner_map || !x || !y || layer >= ctx->cfg.n_layers) return RWTTT_E_INVALID;
  if (n > ctx->cfg.max_group) return RWTTT_E_CAPACITY;
  const uint32_t* owners = owner_map + group->first;
  rwttt_status why = RWTTT_OK;
  if (!ctx->distinct_owners(owners, n, &why)) return why;
  if (!versions_match(ctx, owners, expected ? expected + group->first : nullptr, n))
    return RWTTT_E_STALE_VERSION;
  const int state_bf16 = ctx->cfg.state_dtype == RWTTT_BF16;
  if (rwttt::read_noalloc_bytes(int(ctx->cfg.d_ff), int(ctx->cfg.d_model), state_bf16, int(n)) >
      RWTTT_NOALLOC_SCRATCH_BYTES)
    return RWTTT_E_CAPACITY;

  rwttt::ReadLaunch L;
  L.io_bf16 = ctx->cfg.io_dtype == RWTTT_BF16;
  L.state_bf16 = state_bf16;
  L.d_ff = int(ctx->cfg.d_ff);
  L.d_model = int(ctx->cfg.d_model);
  L.count = int(n);
  L.n_owners = int(ctx->cfg.n_owners);
  L.x = x;
  L.y = y;
  L.w0 = ctx->w0[layer];
  L.workspace = nullptr;
  for (uint32_t b = 0; b < n; ++b) {
    L.dw[b] = ctx->slot(owners[b], layer, 0);
    L.row[b] = owners[b];
    L.tail[b] = nullptr;
  }
  const hipError_t e = rwttt::launch_read_noalloc(L, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(ctx, e);
  return RWTTT_OK;
}

rwttt_status rwttt_attach_tail(rwttt_ctx* ctx, void* const* tail, uint32_t rows) {
  if (!ctx || !tail || rows == 0 || rows > (1u << 20)) return RWTTT_E_INVALID;
  const size_t nl = size_t(ctx->cfg.n_owners) * ctx->cfg.n_layers;
  for (size_t i = 0; i < nl; ++i)
    if (!tail[i] || !aligned16(tail[i])) return RWTTT_E_INVALID;
  ctx->tail.assign(tail, tail + nl);
  ctx->tail_len.assign(nl, 0);
  ctx->tail_rows = rows;
  return RWTTT_OK;
}

rwttt_status rwttt_tail_len(const rwttt_ctx* ctx, uint32_t owner, uint32_t layer, uint32_t* len) {
  if (!ctx || !len || owner >= ctx->cfg.n_owners || layer >= ctx->cfg.n_layers) return RWTTT_E_INVALID;
  *len = ctx->tail.empty() ? 0u : ctx->tail_len[ctx->li(owner, layer)];
  return RWTTT_OK;
}

rwttt_status rwttt_write(rwttt_ctx* ctx, const rwttt_group* group, const uint32_t* owner_map,
                         const uint64_t* expected, uint32_t layer, uint32_t chunk, const void* const* z,
                         const void* const* g, float eta, const void* x, void* y, void* stream) {
  if (!ctx || !group) return RWTTT_E_INVALID;
  if (group->effect != RWTTT_WRITE) return RWTTT_E_KEY_MISMATCH;
  const uint32_t n = group->count;
  if (n == 0) return RWTTT_OK;
  if (!owner_map || !g || layer >= ctx->cfg.n_layers || chunk == 0) return RWTTT_E_INVALID;
  if ((x == nullptr) != (y == nullptr)) return RWTTT_E_INVALID;
  const bool from_tail = z == nullptr;
  if (from_tail && (ctx->tail.empty() || !x || chunk > ctx->tail_rows)) return RWTTT_E_INVALID;
  if (x && (!ctx->cfg.workspace || !aligned16(x) || !aligned16(y))) return RWTTT_E_INVALID;
  if (chunk > (1u << 20)) return RWTTT_E_INVALID;
  if (is_adapter(&ctx->cfg) && chunk > RWTTT_ADAPTER_MAX_CHUNK) return RWTTT_E_INVALID;
  if (n > ctx->cfg.max_group) return RWTTT_E_CAPACITY;
  const uint32_t* owners = owner_map + group->first;
  rwttt_status why = RWTTT_OK;
  if (!ctx->distinct_owners(owners, n, &why)) return why;
  if (!versions_match(ctx, owners, expected ? expected + group->first : nullptr, n))
    return RWTTT_E_STALE_VERSION;
  for (uint32_t b = 0; b < n; ++b) {
    if (!g[b] || !aligned16(g[b])) return RWTTT_E_INVALID;
    if (!from_tail && (!z[b] || !aligned16(z[b]))) return RWTTT_E_INVALID;
    const uint32_t r = owners[b];
    if (from_tail && ctx->tail_len[ctx->li(r, layer)] + 1 != chunk) return RWTTT_E_INVALID;
    if (ctx->failed[r]) return RWTTT_E_WRITE_FAILED;
    if (ctx->written[ctx->li(r, layer)]) return RWTTT_E_DIRTY;
  }
  // a host-only context launches nothing; only an injected failure may open a candidate there
  if (!ctx->cfg.workspace && ctx->inject_failures == 0) return RWTTT_E_INVALID;

  // The write view is open from here until commit or rollback.
  for (uint32_t b = 0; b < n; ++b) {
    const uint32_t r = owners[b];
    ctx->dirty[r] = 1;
    ctx->written[ctx->li(r, layer)] = 1;
  }
  if (ctx->inject_failures > 0) {
    --ctx->inject_failures;
    for (uint32_t b = 0; b < n; ++b) ctx->failed[owners[b]] = 1;
    return RWTTT_E_WRITE_FAILED;
  }

  rwttt::WriteLaunch L;
  L.io_bf16 = ctx->cfg.io_dtype == RWTTT_BF16;
  L.state_bf16 = ctx->cfg.state_dtype == RWTTT_BF16;
  L.d_ff = int(ctx->cfg.d_ff);
  L.d_model = int(ctx->cfg.d_model);
  L.count = int(n);
  L.chunk = int(chunk);
  L.n_owners = int(ctx->cfg.n_owners);
  L.eta = eta;
  L.x = x;
  L.y = y;
  L.w0 = ctx->w0[layer];
  L.workspace = ctx->cfg.workspace;
  for (uint32_t b = 0; b < n; ++b) {
    L.live[b] = ctx->slot(owners[b], layer, 0);
    L.shadow[b] = ctx->slot(owners[b], layer, 1);
    L.z[b] = from_tail ? ctx->tail[ctx->li(owners[b], layer)] : z[b];
    L.g[b] = g[b];
    L.row[b] = owners[b];
  }
  hipError_t e = hipSuccess;
  if (from_tail) {
    // the WRITE step's own input is the chunk's last row
    rwttt::TailLaunch T;
    T.io_bf16 = L.io_bf16;
    T.d_ff = L.d_ff;
    T.count = L.count;
    T.x = x;
    for (uint32_t b = 0; b < n; ++b) {
      T.dst[b] = ctx->tail_row(owners[b], layer, chunk - 1);
      T.row[b] = owners[b];
    }
    e = rwttt::launch_tail_append(T, static_cast<hipStream_t>(stream));
    if (e == hipSuccess)
      for (uint32_t b = 0; b < n; ++b) ctx->tail_len[ctx->li(owners[b], layer)] = chunk;
  }
  if (e == hipSuccess && is_adapter(&ctx->cfg)) {
    if (x) {
      // the step's token at version v, then the factor update
      rwttt::AdapterReadLaunch A;
      A.io_bf16 = L.io_bf16;
      A.state_bf16 = L.state_bf16;
      A.d_ff = L.d_ff;
      A.d_model = L.d_model;
      A.rank = int(ctx->cfg.rank);
      A.count = L.count;
      A.n_owners = L.n_owners;
      A.x = x;
      A.y = y;
      A.w0 = L.w0;
      A.workspace = L.workspace;
      for (uint32_t b = 0; b < n; ++b) {
        A.state[b] = L.live[b];
        A.row[b] = owners[b];
        A.tail[b] = nullptr;
      }
      e = rwttt::launch_adapter_read(A, static_cast<hipStream_t>(stream));
    }
    if (e == hipSuccess) {
      rwttt::AdapterWriteLaunch W;
      W.io_bf16 = L.io_bf16;
      W.state_bf16 = L.state_bf16;
      W.d_ff = L.d_ff;
      W.d_model = L.d_model;
      W.rank = int(ctx->cfg.rank);
      W.count = L.count;
      W.chunk = L.chunk;
      W.n_owners = L.n_owners;
      W.eta = eta;
      W.workspace = L.workspace;
      for (uint32_t b = 0; b < n; ++b) {
        W.live[b] = L.live[b];
        W.shadow[b] = L.shadow[b];
        W.z[b] = L.z[b];
        W.g[b] = L.g[b];
        W.row[b] = owners[b];
      }
      e = rwttt::launch_adapter_write(W, static_cast<hipStream_t>(stream));
    }
  } else if (e == hipSuccess) {
    e = rwttt::launch_write(L, static_cast<hipStream_t>(stream));
  }
  if (e != hipSuccess) {
    for (uint32_t b = 0; b < n; ++b) ctx->failed[owners[b]] = 1;
    return hip_fail(ctx, e);
  }
  return RWTTT_OK;
}

rwttt_status rwttt_commit(rwttt_ctx* ctx, const uint32_t* owners, uint32_t n) {
  if (!ctx || (n && !owners)) return RWTTT_E_INVALID;
  rwttt_status why = RWTTT_OK;
  if (!ctx->distinct_owners(owners, n, &why)) return why;
  for (uint32_t i = 0; i < n; ++i) {
    if (!ctx->dirty[owners[i]]) return RWTTT_E_NOT_DIRTY;
    if (ctx->failed[owners[i]]) return RWTTT_E_WRITE_FAILED;
  }
  for (uint32_t i = 0; i < n; ++i) {
    const uint32_t r = owners[i];
    for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l) {
      const size_t k = ctx->li(r, l);
      if (ctx->written[k]) {
        ctx->live[k] ^= 1;
        ctx->written[k] = 0;
      }
    }
    ctx->version[r] += 1;
    ctx->dirty[r] = 0;
    ctx->clear_tail(r);
  }
  return RWTTT_OK;
}

rwttt_status rwttt_rollback(rwttt_ctx* ctx, const uint32_t* owners, uint32_t n) {
  if (!ctx || (n && !owners)) return RWTTT_E_INVALID;
  rwttt_status why = RWTTT_OK;
  if (!ctx->distinct_owners(owners, n, &why)) return why;
  for (uint32_t i = 0; i < n; ++i)
    if (!ctx->dirty[owners[i]]) return RWTTT_E_NOT_DIRTY;
  for (uint32_t i = 0; i < n; ++i) {
    const uint32_t r = owners[i];
    for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l) ctx->written[ctx->li(r, l)] = 0;
    ctx->dirty[r] = 0;
    ctx->failed[r] = 0;
    ctx->clear_tail(r);
  }
  return RWTTT_OK;
}

rwttt_status rwttt_fork(rwttt_ctx* ctx, uint32_t src, uint32_t dst, void* stream) {
  if (!ctx || src >= ctx->cfg.n_owners || dst >= ctx->cfg.n_owners) return RWTTT_E_INVALID;
  if (src == dst) return RWTTT_E_OWNER_ALIAS;
  if (ctx->dirty[dst]) return RWTTT_E_DIRTY;
  if (!ctx->cfg.workspace) return RWTTT_E_INVALID;
  const size_t state_bytes = slot_bytes_of(&ctx->cfg);
  std::vector<rwttt::CopyJob> jobs;
  for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l) {
    jobs.push_back({ctx->slot(src, l, 0), ctx->slot(dst, l, 0), state_bytes});
    if (!ctx->tail.empty()) {
      const uint32_t rows = ctx->tail_len[ctx->li(src, l)];
      if (rows) jobs.push_back({ctx->tail[ctx->li(src, l)], ctx->tail[ctx->li(dst, l)],
                                size_t(rows) * ctx->cfg.d_ff * ctx->io_bytes()});
    }
  }
  const hipError_t e = rwttt::launch_copy(jobs.data(), int(jobs.size()),
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(ctx, e);
  ctx->version[dst] = ctx->version[src];
  ctx->failed[dst] = 0;
  if (!ctx->tail.empty())
    for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l)
      ctx->tail_len[ctx->li(dst, l)] = ctx->tail_len[ctx->li(src, l)];
  return RWTTT_OK;
}

rwttt_status rwttt_checkpoint(rwttt_ctx* ctx, uint32_t owner, void* const* dst, uint64_t* version,
                              void* stream) {
  if (!ctx || !dst || !version || owner >= ctx->cfg.n_owners) return RWTTT_E_INVALID;
  if (!ctx->cfg.workspace) return RWTTT_E_INVALID;   // host-only context: no device copies
  for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l)
    if (!dst[l]) return RWTTT_E_INVALID;
  const size_t state_bytes = slot_bytes_of(&ctx->cfg);
  for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l) {
    const hipError_t e = hipMemcpyAsync(dst[l], ctx->slot(owner, l, 0), state_bytes,
                                        hipMemcpyDefault, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(ctx, e);
  }
  *version = ctx->version[owner];
  return RWTTT_OK;
}

rwttt_status rwttt_resume(rwttt_ctx* ctx, uint32_t owner, const void* const* src, uint64_t version,
                          void* stream) {
  if (!ctx || !src || owner >= ctx->cfg.n_owners) return RWTTT_E_INVALID;
  if (ctx->dirty[owner]) return RWTTT_E_DIRTY;
  if (!ctx->cfg.workspace) return RWTTT_E_INVALID;   // host-only context: no device copies
  for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l)
    if (!src[l]) return RWTTT_E_INVALID;
  const size_t state_bytes = slot_bytes_of(&ctx->cfg);
  for (uint32_t l = 0; l < ctx->cfg.n_layers; ++l) {
    const hipError_t e = hipMemcpyAsync(ctx->slot(owner, l, 0), src[l], state_bytes,
                                        hipMemcpyDefault, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(ctx, e);
  }
  ctx->version[owner] = version;
  ctx->clear_tail(owner);
  return RWTTT_OK;
}

rwttt_status rwttt_version(const rwttt_ctx* ctx, uint32_t owner, uint64_t* version, int32_t* dirty) {
  if (!ctx || owner >= ctx->cfg.n_owners) return RWTTT_E_INVALID;
  if (version) *version = ctx->version[owner];
  if (dirty) *dirty = ctx->dirty[owner];
  return RWTTT_OK;
}

rwttt_status rwttt_slot(const rwttt_ctx* ctx, uint32_t owner, uint32_t layer, int32_t which,
                        void** ptr) {
  if (!ctx || !ptr || owner >= ctx->cfg.n_owners || layer >= ctx->cfg.n_layers) return RWTTT_E_INVALID;
  if (which != 0 && which != 1) return RWTTT_E_INVALID;
  *ptr = ctx->slot(owner, layer, which);
  return RWTTT_OK;
}

rwttt_status rwttt_inject_write_failures(rwttt_ctx* ctx, uint32_t count) {
  if (!ctx) return RWTTT_E_INVALID;
  ctx->inject_failures = count;
  return RWTTT_OK;
}

int32_t rwttt_last_hip_error(const rwttt_ctx* ctx) { return ctx ? ctx->last_hip : 0; }

const char* rwttt_strerror(rwttt_status s) {
  switch (s) {
    case RWTTT_OK: return "ok";
    case RWTTT_DEFERRED: return "deferred by the wait budget";
    case RWTTT_E_INVALID: return "invalid argument";
    case RWTTT_E_STALE_VERSION: return "expected version differs from the committed version";
    case RWTTT_E_OWNER_ALIAS: return "owner named twice";
    case RWTTT_E_KEY_MISMATCH: return "wrong effect for this call";
    case RWTTT_E_NOT_DIRTY: return "owner has no open candidate";
    case RWTTT_E_DIRTY: return "owner already holds an uncommitted candidate";
    case RWTTT_E_CAPACITY: return "output array or workspace too small";
    case RWTTT_E_HIP: return "HIP launch or runtime error";
    case RWTTT_E_WRITE_FAILED: return "the owner's WRITE failed; roll it back";
    default: return "unknown status";
  }
}

}  // extern "C"
