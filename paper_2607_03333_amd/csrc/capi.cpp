// C ABI of libspork (declared in include/spork.h): argument checks, error
// reporting, block-manager and planner calls, kernel dispatch.
#include "spork.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "block_manager.h"
#include "ceiling_kernels.h"
#include "kernels.h"
#include "ngram_kernels.h"
#include "noalloc.h"
#include "vocab_kernels.h"
#include "plan.h"

struct spork_cache {
  spork::BlockManager bm;
  spork_cache(int32_t nb, int32_t bs, const int32_t* order) : bm(nb, bs, order) {}
};

struct spork_plan {
  spork::Plan p;
  spork_shape shape;
};

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

constexpr int kAbiVersion = 2;

// Per-thread kernel timing: event pairs recorded around each launch.
struct Timing {
  bool on = false;
  std::vector<hipEvent_t> pool;  // created lazily, reused across reads
  size_t used = 0;
  std::vector<std::pair<int, size_t>> marks;  // (kind, index of the begin event)
};
thread_local Timing g_timing;

hipEvent_t next_event() {
  if (g_timing.used == g_timing.pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_timing.pool.push_back(e);
  }
  return g_timing.pool[g_timing.used++];
}

// Launch `f` on `stream`, bracketed by timing events of `kind` when enabled.
template <typename F>
hipError_t timed(int kind, hipStream_t stream, F&& f) {
  if (!g_timing.on) return f();
  const size_t at = g_timing.used;
  hipEvent_t b = next_event(), e = next_event();
  if (b == nullptr || e == nullptr) return hipErrorOutOfMemory;
  hipError_t rc = hipEventRecord(b, stream);
  if (rc != hipSuccess) return rc;
  rc = f();
  if (rc != hipSuccess) return rc;
  rc = hipEventRecord(e, stream);
  if (rc == hipSuccess) g_timing.marks.push_back({kind, at});
  return rc;
}

int from_bm(spork::BmStatus s, const char* what) {
  switch (s) {
    case spork::BmStatus::kOk: return SPORK_OK;
    case spork::BmStatus::kUnknownSeq: return fail(SPORK_E_INVAL, std::string(what) + ": unknown sequence id");
    case spork::BmStatus::kBadArg: return fail(SPORK_E_INVAL, std::string(what) + ": bad argument");
    case spork::BmStatus::kNoBlocks: return fail(SPORK_E_NOBLOCKS, std::string(what) + ": not enough free blocks");
  }
  return fail(SPORK_E_INVAL, what);
}

int elem_bytes(int32_t dtype) { return dtype == SPORK_DTYPE_BF16 ? 2 : (dtype == SPORK_DTYPE_F32 ? 4 : 0); }

int check_shape(const spork_shape* sh) {
  if (sh == nullptr) return fail(SPORK_E_INVAL, "shape is NULL");
  if (sh->hq <= 0 || sh->hkv <= 0 || sh->hq % sh->hkv != 0)
    return fail(SPORK_E_INVAL, "hq and hkv must be positive and hq a multiple of hkv");
  if (sh->head_dim <= 0 || sh->block_size <= 0) return fail(SPORK_E_INVAL, "head_dim and block_size must be positive");
  if (elem_bytes(sh->dtype) == 0) return fail(SPORK_E_UNSUPPORTED, "dtype must be SPORK_DTYPE_F32 or SPORK_DTYPE_BF16");
  if (!std::isfinite(sh->sm_scale)) return fail(SPORK_E_INVAL, "sm_scale must be finite");
  return SPORK_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <typename F>
int guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return fail(SPORK_E_INVAL, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(SPORK_E_INVAL, e.what());
  } catch (...) {
    return fail(SPORK_E_INVAL, "unknown error");
  }
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SPORK_OK;
  return fail(SPORK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

extern "C" {

const char* spork_last_error(void) { return g_last_error.c_str(); }

int spork_version(void) { return kAbiVersion; }

int spork_cache_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                       spork_cache** out) {
  return guarded([&] {
    if (out == nullptr) return fail(SPORK_E_INVAL, "out is NULL");
    if (num_blocks <= 0 || block_size <= 0) return fail(SPORK_E_INVAL, "num_blocks and block_size must be positive");
    if (free_order != nullptr) {
      std::string seen(static_cast<size_t>(num_blocks), '\0');
      for (int32_t i = 0; i < num_blocks; ++i) {
        const int32_t b = free_order[i];
        if (b < 0 || b >= num_blocks || seen[b]) return fail(SPORK_E_INVAL, "free_order is not a permutation");
        seen[b] = 1;
      }
    }
    *out = new spork_cache(num_blocks, block_size, free_order);
    return SPORK_OK;
  });
}

int spork_cache_destroy(spork_cache* cache) {
  delete cache;
  return SPORK_OK;
}

int spork_seq_new(spork_cache* cache, int32_t* seq_out) {
  return guarded([&] {
    if (cache == nullptr || seq_out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
    *seq_out = cache->bm.seq_new();
    return SPORK_OK;
  });
}

int spork_seq_append(spork_cache* cache, int32_t seq, int32_t n_tokens, int64_t* slots_out,
                     int32_t* cow_out, int32_t* n_cow_out) {
  return guarded([&] {
    if (cache == nullptr || cow_out == nullptr || n_cow_out == nullptr || (n_tokens > 0 && slots_out == nullptr))
      return fail(SPORK_E_INVAL, "NULL argument");
    spork::CowCopy cow;
    int32_t n_cow = 0;
    const int rc = from_bm(cache->bm.append(seq, n_tokens, slots_out, &cow, &n_cow), "spork_seq_append");
    if (rc != SPORK_OK) return rc;
    *n_cow_out = n_cow;
    cow_out[0] = cow.src;
    cow_out[1] = cow.dst;
    cow_out[2] = cow.n_valid;
    return SPORK_OK;
  });
}

int spork_seq_append_batch(spork_cache* cache, const int32_t* seqs, const int32_t* n_tokens, int32_t n_seqs,
                           int64_t* slots_out, int32_t* cow_out, int32_t* n_cow_out) {
  return guarded([&] {
    if (cache == nullptr || n_cow_out == nullptr || n_seqs < 0) return fail(SPORK_E_INVAL, "NULL argument or n_seqs < 0");
    if (n_seqs > 0 && (seqs == nullptr || n_tokens == nullptr || cow_out == nullptr))
      return fail(SPORK_E_INVAL, "NULL argument");
    int64_t total = 0;
    for (int32_t i = 0; i < n_seqs; ++i) total += n_tokens[i] > 0 ? n_tokens[i] : 0;
    if (total > 0 && slots_out == nullptr) return fail(SPORK_E_INVAL, "slots_out is NULL");
    std::vector<spork::CowCopy> cows(static_cast<size_t>(n_seqs));
    int32_t n_cow = 0;
    const int rc = from_bm(cache->bm.append_batch(seqs, n_tokens, n_seqs, slots_out, cows.data(), &n_cow),
                           "spork_seq_append_batch");
    if (rc != SPORK_OK) return rc;
    for (int32_t i = 0; i < n_cow; ++i) {
      cow_out[3 * i] = cows[i].src;
      cow_out[3 * i + 1] = cows[i].dst;
      cow_out[3 * i + 2] = cows[i].n_valid;
    }
    *n_cow_out = n_cow;
    return SPORK_OK;
  });
}

int spork_fork(spork_cache* cache, int32_t parent_seq, int32_t* child_seq_out) {
  return guarded([&] {
    if (cache == nullptr || child_seq_out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
    return from_bm(cache->bm.fork(parent_seq, child_seq_out), "spork_fork");
  });
}

int spork_seq_free(spork_cache* cache, int32_t seq) {
  return guarded([&] {
    if (cache == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
    return from_bm(cache->bm.free_seq(seq), "spork_seq_free");
  });
}

int spork_seq_len(const spork_cache* cache, int32_t seq, int32_t* len_out) {
  if (cache == nullptr || len_out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  if (!cache->bm.has(seq)) return fail(SPORK_E_INVAL, "spork_seq_len: unknown sequence id");
  *len_out = cache->bm.length(seq);
  return SPORK_OK;
}

int spork_block_table(const spork_cache* cache, int32_t seq, int32_t* out, int32_t cap, int32_t* n_out) {
  if (cache == nullptr || n_out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  if (!cache->bm.has(seq)) return fail(SPORK_E_INVAL, "spork_block_table: unknown sequence id");
  const auto& t = cache->bm.table(seq);
  *n_out = static_cast<int32_t>(t.size());
  if (static_cast<int64_t>(t.size()) > cap) return fail(SPORK_E_CAPACITY, "spork_block_table: out too small");
  if (!t.empty()) {
    if (out == nullptr) return fail(SPORK_E_INVAL, "out is NULL");
    std::memcpy(out, t.data(), t.size() * sizeof(int32_t));
  }
  return SPORK_OK;
}

int spork_refcount(const spork_cache* cache, int32_t block, int32_t* out) {
  if (cache == nullptr || out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  if (block < 0 || block >= cache->bm.num_blocks()) return fail(SPORK_E_INVAL, "block out of range");
  *out = cache->bm.refcount(block);
  return SPORK_OK;
}

int spork_free_blocks(const spork_cache* cache, int32_t* out, int32_t cap, int32_t* n_out) {
  if (cache == nullptr || n_out == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  const auto& q = cache->bm.free_queue();
  *n_out = static_cast<int32_t>(q.size());
  if (static_cast<int64_t>(q.size()) > cap) return fail(SPORK_E_CAPACITY, "spork_free_blocks: out too small");
  if (!q.empty() && out == nullptr) return fail(SPORK_E_INVAL, "out is NULL");
  int32_t i = 0;
  for (int32_t b : q) out[i++] = b;
  return SPORK_OK;
}

int spork_kv_write(const spork_shape* shape, void* k_cache, void* v_cache, int32_t num_blocks,
                   const int64_t* slots, const void* k_new, const void* v_new, int32_t n,
                   int32_t* bad_slots, hipStream_t stream) {
  return guarded([&] {
    int rc = check_shape(shape);
    if (rc != SPORK_OK) return rc;
    if (n < 0 || num_blocks <= 0) return fail(SPORK_E_INVAL, "n must be >= 0 and num_blocks > 0");
    if (n == 0) return SPORK_OK;
    if (!k_cache || !v_cache || !slots || !k_new || !v_new) return fail(SPORK_E_INVAL, "NULL pointer");
    const int vec = 16 / elem_bytes(shape->dtype);
    if (shape->head_dim % vec != 0) return fail(SPORK_E_UNSUPPORTED, "head_dim must fill 16-byte vectors");
    if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) || !aligned16(v_new))
      return fail(SPORK_E_INVAL, "pools and token arrays must be 16-byte aligned");
    const int64_t num_slots = static_cast<int64_t>(num_blocks) * shape->block_size;
    return hip_status(spork::launch_kv_write(shape->dtype, shape->hkv, shape->head_dim, shape->block_size,
                                             num_slots, k_cache, v_cache, slots, k_new, v_new, n, bad_slots,
                                             stream),
                      "spork_kv_write");
  });
}

int spork_kv_copy(const spork_shape* shape, void* k_cache, void* v_cache, int32_t num_blocks,
                  int32_t src_block, int32_t dst_block, int32_t n_valid, hipStream_t stream) {
  return guarded([&] {
    int rc = check_shape(shape);
    if (rc != SPORK_OK) return rc;
    if (!k_cache || !v_cache) return fail(SPORK_E_INVAL, "NULL pointer");
    if (src_block < 0 || src_block >= num_blocks || dst_block < 0 || dst_block >= num_blocks || src_block == dst_block)
      return fail(SPORK_E_INVAL, "src/dst block out of range or equal");
    if (n_valid < 0 || n_valid > shape->block_size) return fail(SPORK_E_INVAL, "n_valid out of range");
    return hip_status(spork::launch_kv_copy(shape->dtype, shape->hkv, shape->head_dim, shape->block_size, k_cache,
                                            v_cache, src_block, dst_block, n_valid, stream),
                      "spork_kv_copy");
  });
}

int spork_plan_create(const spork_cache* cache, const spork_shape* shape, const int32_t* seqs,
                      const int32_t* n_rows, const int32_t* groups, int32_t n_threads, int32_t n_cu,
                      spork_plan** out) {
  return guarded([&] {
    if (cache == nullptr || out == nullptr || seqs == nullptr || n_rows == nullptr || groups == nullptr)
      return fail(SPORK_E_INVAL, "NULL argument");
    int rc = check_shape(shape);
    if (rc != SPORK_OK) return rc;
    // bf16: persistent 4-wave workgroups with up to 2 row tiles per wave, two
    // per compute unit (68 KB of LDS each). When some range has more than 8
    // row tiles (verify at K = 16 and more, multi-row probe prefill), 4-wave
    // workgroups would stream that range once per row slice: the batch is
    // planned again for one 8-wave workgroup per compute unit (up to 16
    // tiles in one slice, an 8-stage 128 KB ring). fp32: one 1-wave
    // workgroup per unit with up to 4 row tiles, 4 per CU (8 with up to 2).
    const bool bf16 = shape->dtype == SPORK_DTYPE_BF16;
    auto shape_for = [&](int32_t waves) {
      return spork::PlanShape{shape->hq, shape->hkv, shape->head_dim, shape->block_size, elem_bytes(shape->dtype),
                              bf16 ? 2 * waves : 4, bf16 ? 8 / waves : 4, bf16 ? 8 / waves : 8, bf16,
                              bf16 ? waves : 1};
    };
    auto* plan = new spork_plan();
    plan->shape = *shape;
    std::string err = spork::build_plan(cache->bm, shape_for(4), seqs, n_rows, groups, n_threads, n_cu, &plan->p);
    if (err.empty() && bf16 && plan->p.max_range_tiles > 8) {
      plan->p = spork::Plan{};
      err = spork::build_plan(cache->bm, shape_for(8), seqs, n_rows, groups, n_threads, n_cu, &plan->p);
    }
    if (!err.empty()) {
      delete plan;
      return fail(SPORK_E_INVAL, "spork_plan_create: " + err);
    }
    *out = plan;
    return SPORK_OK;
  });
}

int spork_plan_destroy(spork_plan* plan) {
  delete plan;
  return SPORK_OK;
}

int spork_plan_get_info(const spork_plan* plan, spork_plan_info* info) {
  if (plan == nullptr || info == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  const spork::Plan& p = plan->p;
  std::memset(info, 0, sizeof(*info));
  info->n_threads = p.n_threads;
  info->n_rows = p.n_rows;
  info->n_groups = p.n_groups;
  info->n_items = p.n_items;
  info->n_units = p.n_units;
  info->attn_grid = p.grid;
  info->n_partials = p.n_partials;
  info->max_row_tiles = p.row_tiles;
  info->attn_waves = p.shape.waves;
  info->image_bytes = p.image.size();
  info->workspace_bytes = p.workspace_bytes;
  info->shared_tokens = p.shared_tokens;
  info->private_tokens = p.private_tokens;
  const int64_t per_tok = 2LL * p.shape.hkv * p.shape.head_dim * p.shape.elem_bytes;
  info->unique_kv_bytes = (p.shared_tokens + p.private_tokens) * per_tok;
  info->flat_kv_bytes = p.flat_tokens * per_tok;
  info->control_bytes = p.control_bytes;
  return SPORK_OK;
}

int spork_plan_advance(spork_plan* plan, const spork_cache* cache, void* dev_image, hipStream_t stream) {
  return guarded([&] {
    if (plan == nullptr || cache == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
    spork::Plan& p = plan->p;
    const spork::BlockManager& bm = cache->bm;
    if (dev_image == nullptr || (reinterpret_cast<uintptr_t>(dev_image) & 255) != 0)
      return fail(SPORK_E_INVAL, "dev_image must be non-NULL and 256-byte aligned");
    if (bm.block_size() != p.shape.block_size) return fail(SPORK_E_INVAL, "cache block size differs from the plan's");
    const size_t n = p.seqs.size();
    std::vector<int32_t> g(n, 0);
    // Every check first: on an error nothing is launched and the plan is unchanged.
    for (size_t t = 0; t < n; ++t) {
      const int32_t seq = p.seqs[t];
      if (!bm.has(seq)) return fail(SPORK_E_INVAL, "spork_plan_advance: a planned sequence was freed; plan again");
      g[t] = bm.length(seq) - p.len[t];
      if (g[t] < 0) return fail(SPORK_E_INVAL, "spork_plan_advance: a sequence is shorter than planned; plan again");
      if (g[t] > 0 && p.thread_items[t].empty())
        return fail(SPORK_E_CAPACITY, "spork_plan_advance: a grown thread has no private range to extend; plan again");
      if (p.thread_table_off[t] >= 0) {
        // The block manager changes a live table only by appending entries
        // and by copying the block an append writes into, the last one: the
        // planned entries are unchanged when the last of them is.
        const auto& cur = bm.table(seq);
        const auto& have = p.thread_table[t];
        if (cur.size() < have.size() || (!have.empty() && cur[have.size() - 1] != have.back()))
          return fail(SPORK_E_INVAL, "spork_plan_advance: planned blocks changed (copy-on-write or free); plan again");
        if (static_cast<int64_t>(cur.size()) > p.thread_table_cap[t])
          return fail(SPORK_E_CAPACITY, "spork_plan_advance: more new blocks than the plan reserves; plan again");
      }
    }
    const auto* waves = reinterpret_cast<const spork::WaveDesc*>(p.image.data() + p.off_waves);
    auto* items = reinterpret_cast<spork::ItemDesc*>(p.image.data() + p.off_items);
    for (int32_t u : p.open_units) {
      const spork::WaveDesc& w = waves[u];
      const int32_t t = items[w.item].thread;
      if (spork::unit_table_span(w.tok_lo, w.tok_hi + g[t], p.shape.block_size) > spork::kUnitTableEntries)
        return fail(SPORK_E_CAPACITY, "spork_plan_advance: a private range outgrew its unit; plan again");
    }
    // Patches: each grown thread's `grow` in its private items, the new
    // entries of its table; written into the host image too.
    std::vector<std::pair<int32_t, int32_t>> patch;
    auto* words = reinterpret_cast<int32_t*>(p.image.data());
    const int32_t items_w = static_cast<int32_t>(p.off_items / 4), tables_w = static_cast<int32_t>(p.off_tables / 4);
    int64_t added = 0;
    for (size_t t = 0; t < n; ++t) {
      if (g[t] != p.grow[t]) {
        for (int32_t i : p.thread_items[t]) patch.push_back({items_w + i * 8 + 6, g[t]});
        added += g[t] - p.grow[t];
      }
      if (p.thread_table_off[t] >= 0) {
        const auto& cur = bm.table(p.seqs[t]);
        for (size_t k = p.thread_table[t].size(); k < cur.size(); ++k)
          patch.push_back({tables_w + p.thread_table_off[t] + static_cast<int32_t>(k), cur[k]});
      }
    }
    for (size_t i = 0; i < patch.size(); i += spork::kPatchMax) {
      spork::ImagePatch ip{};
      ip.n = static_cast<int32_t>(std::min<size_t>(spork::kPatchMax, patch.size() - i));
      for (int32_t k = 0; k < ip.n; ++k) {
        ip.off[k] = patch[i + k].first;
        ip.val[k] = patch[i + k].second;
      }
      const int rc = hip_status(spork::launch_image_patch(static_cast<int32_t*>(dev_image), ip, stream),
                                "spork_plan_advance");
      if (rc != SPORK_OK) return rc;  // earlier patches of this call may have run; plan again
    }
    for (const auto& pw : patch) words[pw.first] = pw.second;
    for (size_t t = 0; t < n; ++t) {
      p.grow[t] = g[t];
      if (p.thread_table_off[t] >= 0) {
        const auto& cur = bm.table(p.seqs[t]);
        p.thread_table[t].insert(p.thread_table[t].end(), cur.begin() + p.thread_table[t].size(), cur.end());
      }
    }
    p.private_tokens += added;
    p.flat_tokens += added;
    return SPORK_OK;
  });
}

int spork_plan_image(const spork_plan* plan, void* host_dst, size_t cap) {
  if (plan == nullptr || host_dst == nullptr) return fail(SPORK_E_INVAL, "NULL argument");
  if (cap < plan->p.image.size()) return fail(SPORK_E_CAPACITY, "spork_plan_image: destination too small");
  std::memcpy(host_dst, plan->p.image.data(), plan->p.image.size());
  return SPORK_OK;
}

int spork_workspace_clear(const spork_plan* plan, void* workspace, size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    if (plan == nullptr) return fail(SPORK_E_INVAL, "plan is NULL");
    const size_t n = plan->p.control_bytes;
    if (n == 0) return SPORK_OK;
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
      return fail(SPORK_E_INVAL, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < n) return fail(SPORK_E_CAPACITY, "workspace smaller than info.control_bytes");
    return hip_status(spork::launch_counter_reset(static_cast<int32_t*>(workspace), static_cast<int32_t>(n / 4), stream),
                      "spork_workspace_clear");
  });
}

// Attention over a plan. bf16 (persistent): the attention launch (with the
// argmax units of a verify step in its tail), then the merge launch (with
// the accept). fp32: the argmax first (verify), the attention, the merge.
// Checks of the attention arguments that come before anything is launched.
static int check_attention(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                           const void* v_cache, const void* out) {
  const spork::Plan& p = plan->p;
  const spork_shape& sh = plan->shape;
  if (!spork::attention_supported(sh.dtype, sh.head_dim, sh.block_size, p.row_tiles, p.shape.waves))
    return fail(SPORK_E_UNSUPPORTED, "no attention kernel for this dtype / head_dim / block_size / row tiles "
                                     "(bf16: head_dim 128; f32: head_dim 64 or 128; block_size 16 or 32)");
  if (!dev_image || !q || !k_cache || !v_cache || !out) return fail(SPORK_E_INVAL, "NULL pointer");
  if ((reinterpret_cast<uintptr_t>(dev_image) & 255) != 0) return fail(SPORK_E_INVAL, "dev_image must be 256-byte aligned");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
    return fail(SPORK_E_INVAL, "q, pools and out must be 16-byte aligned");
  return SPORK_OK;
}

static int attention(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                     const void* v_cache, void* out, float* lse, void* workspace, size_t ws_bytes,
                     const spork::AcceptArgs* acc, hipStream_t stream) {
  const spork::Plan& p = plan->p;
  const spork_shape& sh = plan->shape;
  int rc0 = check_attention(plan, dev_image, q, k_cache, v_cache, out);
  if (rc0 != SPORK_OK) return rc0;
  if (ws_bytes < p.workspace_bytes) return fail(SPORK_E_CAPACITY, "workspace smaller than info.workspace_bytes");
  if (p.workspace_bytes > 0 && (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0))
    return fail(SPORK_E_INVAL, "workspace must be non-NULL and 256-byte aligned");
  const auto* img = static_cast<const uint8_t*>(dev_image);
  spork::AttnArgs a{};
  a.waves = reinterpret_cast<const spork::WaveDesc*>(img + p.off_waves);
  a.items = reinterpret_cast<const spork::ItemDesc*>(img + p.off_items);
  a.rows = reinterpret_cast<const spork::RowDesc*>(img + p.off_rows);
  a.tables = reinterpret_cast<const int32_t*>(img + p.off_tables);
  a.merge_off = reinterpret_cast<const int32_t*>(img + p.off_merge_off);
  a.part_slot = reinterpret_cast<const int32_t*>(img + p.off_part_slot);
  a.wg_off = reinterpret_cast<const int32_t*>(img + p.off_wg_off);
  a.cursors = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(workspace) + p.off_ws_cursors);
  a.n_units = p.n_units;
  a.grid = p.grid;
  a.n_lists = p.n_lists;
  a.n_out = p.n_out;
  a.row_tiles = p.row_tiles;
  a.wg_waves = p.shape.waves;
  a.hq = sh.hq;
  a.hkv = sh.hkv;
  a.head_dim = sh.head_dim;
  a.block_size = sh.block_size;
  a.dtype = sh.dtype;
  a.scale_log2 = sh.sm_scale * 1.4426950408889634f;
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.out = out;
  a.lse = lse;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.part_o = ws + p.off_ws_o;
  a.part_ml = reinterpret_cast<float*>(ws + p.off_ws_ml);
  a.n_cursors = p.n_cursors;
  // The persistent bf16 kernel takes its units through cursors that are zero
  // on entry (the merge launch clears them again); in a verify step it also
  // runs the argmax units after its lists, and the accept rides in the merge
  // launch: two launches. The fp32 kernel is not persistent: the argmax has
  // a launch of its own first.
  const bool persistent = p.shape.persistent;
  const bool verify = acc != nullptr && acc->n_verify > 0;
  int rc = SPORK_OK;
  if (verify) a.acc = *acc;
  if (persistent) {
    if (verify) a.tail_units = acc->n_verify * (acc->k_drafts + 1) * acc->chunks;
  } else if (verify) {
    rc = hip_status(timed(SPORK_KERNEL_ARGMAX, stream, [&] { return spork::launch_argmax(a.acc, stream); }),
                    "spork_verify_accept (argmax)");
  }
  if (rc != SPORK_OK) return rc;
  rc = hip_status(timed(SPORK_KERNEL_ATTN, stream, [&] { return spork::launch_attn_partial(a, stream); }),
                  "spork_attn_decode (partial attention)");
  if (rc != SPORK_OK) return rc;
  return hip_status(timed(SPORK_KERNEL_MERGE, stream, [&] { return spork::launch_merge(a, stream); }),
                    "spork_attn_decode (merge)");
}

int spork_attn_decode(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                      const void* v_cache, void* out, float* lse, void* workspace, size_t ws_bytes,
                      hipStream_t stream) {
  return guarded([&] {
    if (plan == nullptr) return fail(SPORK_E_INVAL, "plan is NULL");
    return attention(plan, dev_image, q, k_cache, v_cache, out, lse, workspace, ws_bytes, nullptr, stream);
  });
}

int spork_verify_workspace_bytes(int32_t n_verify, int32_t k_drafts, int32_t vocab, size_t* bytes) {
  if (bytes == nullptr) return fail(SPORK_E_INVAL, "bytes is NULL");
  if (n_verify < 0 || k_drafts < 0 || vocab <= 0) return fail(SPORK_E_INVAL, "bad sizes");
  const int32_t rows = n_verify * (k_drafts + 1);
  *bytes = static_cast<size_t>(rows) * spork::accept_chunks(rows, vocab) * sizeof(uint64_t);
  return SPORK_OK;
}

}  // extern "C"

// The verify step over a caller's workspace, or (scratch = true) over the
// library's per-device scratch array, in which case `workspace` and
// `ws_bytes` are ignored.
static int verify_accept(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                         const void* v_cache, void* out, float* lse, const void* logits, int32_t logits_dtype,
                         int32_t vocab, const int32_t* drafts, int32_t n_verify, int32_t k_drafts,
                         int32_t* accept_len, int32_t* next_token, int32_t* argmax_out, void* workspace,
                         size_t ws_bytes, bool scratch, hipStream_t stream) {
  return guarded([&] {
    if (n_verify < 0 || k_drafts < 0 || k_drafts > 4096 || vocab <= 0)
      return fail(SPORK_E_INVAL, "n_verify >= 0, 0 <= k_drafts <= 4096 and vocab > 0 required");
    if (logits_dtype != SPORK_DTYPE_F32 && logits_dtype != SPORK_DTYPE_BF16)
      return fail(SPORK_E_UNSUPPORTED, "logits dtype must be f32 or bf16");
    const int64_t rows = static_cast<int64_t>(n_verify) * (k_drafts + 1);
    if (rows * static_cast<int64_t>(vocab) > (static_cast<int64_t>(1) << 40)) return fail(SPORK_E_INVAL, "logits too large");
    if (n_verify > 0 && (!logits || !accept_len || !next_token || (k_drafts > 0 && !drafts)))
      return fail(SPORK_E_INVAL, "NULL pointer");
    size_t att_ws = 0;
    if (plan != nullptr) att_ws = (plan->p.workspace_bytes + 255) & ~static_cast<size_t>(255);
    size_t acc_ws = 0;
    spork_verify_workspace_bytes(n_verify, k_drafts, vocab, &acc_ws);
    if (scratch) {
      if (att_ws + acc_ws > spork::kScratchBytes)
        return fail(SPORK_E_CAPACITY, "spork_verify_accept_noalloc: the step needs " + std::to_string(att_ws + acc_ws) +
                                          " bytes of scratch, more than the library's " +
                                          std::to_string(spork::kScratchBytes) + " (use spork_verify_accept)");
      if (plan != nullptr) {
        const int rc = check_attention(plan, dev_image, q, k_cache, v_cache, out);
        if (rc != SPORK_OK) return rc;
      }
      const int rc = hip_status(spork::scratch_acquire(plan != nullptr ? plan->p.control_bytes : 0, stream, &workspace),
                                "spork_verify_accept_noalloc (scratch)");
      if (rc != SPORK_OK) return rc;
      ws_bytes = spork::kScratchBytes;
    }
    if (ws_bytes < att_ws + acc_ws) return fail(SPORK_E_CAPACITY, "workspace too small for attention + accept");
    if ((att_ws + acc_ws) > 0 && (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0))
      return fail(SPORK_E_INVAL, "workspace must be non-NULL and 256-byte aligned");
    spork::AcceptArgs a{};
    a.logits = logits;
    a.logits_dtype = logits_dtype;
    a.vocab = vocab;
    a.n_verify = n_verify;
    a.k_drafts = k_drafts;
    a.chunks = spork::accept_chunks(static_cast<int32_t>(rows), vocab);
    a.drafts = drafts;
    a.accept_len = accept_len;
    a.next_token = next_token;
    a.argmax_out = argmax_out;
    a.keys = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(workspace) + att_ws);
    if (plan != nullptr)
      return attention(plan, dev_image, q, k_cache, v_cache, out, lse, workspace, ws_bytes, &a, stream);
    if (n_verify == 0) return SPORK_OK;
    const int rc = hip_status(timed(SPORK_KERNEL_ARGMAX, stream, [&] { return spork::launch_argmax(a, stream); }),
                              "spork_verify_accept (argmax)");
    if (rc != SPORK_OK) return rc;
    return hip_status(timed(SPORK_KERNEL_ACCEPT, stream, [&] { return spork::launch_accept_tail(a, stream); }),
                      "spork_verify_accept (accept)");
  });
}

extern "C" {

int spork_verify_accept(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                        const void* v_cache, void* out, float* lse, const void* logits, int32_t logits_dtype,
                        int32_t vocab, const int32_t* drafts, int32_t n_verify, int32_t k_drafts,
                        int32_t* accept_len, int32_t* next_token, int32_t* argmax_out, void* workspace,
                        size_t ws_bytes, hipStream_t stream) {
  return verify_accept(plan, dev_image, q, k_cache, v_cache, out, lse, logits, logits_dtype, vocab, drafts, n_verify,
                       k_drafts, accept_len, next_token, argmax_out, workspace, ws_bytes, false, stream);
}

int spork_verify_accept_noalloc(const spork_plan* plan, const void* dev_image, const void* q, const void* k_cache,
                                const void* v_cache, void* out, float* lse, const void* logits,
                                int32_t logits_dtype, int32_t vocab, const int32_t* drafts, int32_t n_verify,
                                int32_t k_drafts, int32_t* accept_len, int32_t* next_token, int32_t* argmax_out,
                                hipStream_t stream) {
  // No timing events here: creating one may allocate.
  const bool timing = g_timing.on;
  g_timing.on = false;
  const int rc = verify_accept(plan, dev_image, q, k_cache, v_cache, out, lse, logits, logits_dtype, vocab, drafts,
                               n_verify, k_drafts, accept_len, next_token, argmax_out, nullptr, 0, true, stream);
  g_timing.on = timing;
  return rc;
}

int spork_confidence_workspace_bytes(int32_t n_rows, int32_t vocab, size_t* bytes) {
  if (bytes == nullptr) return fail(SPORK_E_INVAL, "bytes is NULL");
  if (n_rows < 0 || vocab <= 0) return fail(SPORK_E_INVAL, "n_rows >= 0 and vocab > 0 required");
  // per (row, chunk): the argmax key and the (max, sum) pair
  *bytes = static_cast<size_t>(n_rows) * spork::accept_chunks(n_rows, vocab) * (sizeof(uint64_t) + 2 * sizeof(float));
  return SPORK_OK;
}

int spork_probe_confidence(const void* logits, int32_t logits_dtype, int32_t vocab, int32_t n_rows,
                           const int32_t* span_off, int32_t n_probes, float theta, int32_t* argmax_out,
                           float* logprob_out, float* confidence_out, int32_t* commit_out, void* workspace,
                           size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    if (n_rows < 0 || n_probes < 0 || vocab <= 0)
      return fail(SPORK_E_INVAL, "n_rows >= 0, n_probes >= 0 and vocab > 0 required");
    if (logits_dtype != SPORK_DTYPE_F32 && logits_dtype != SPORK_DTYPE_BF16)
      return fail(SPORK_E_UNSUPPORTED, "logits dtype must be f32 or bf16");
    if (static_cast<int64_t>(n_rows) * vocab > (static_cast<int64_t>(1) << 40))
      return fail(SPORK_E_INVAL, "logits too large");
    if (n_rows > 0 && logits == nullptr) return fail(SPORK_E_INVAL, "logits is NULL");
    if (n_probes > 0 && (span_off == nullptr || confidence_out == nullptr))
      return fail(SPORK_E_INVAL, "span_off and confidence_out are required when n_probes > 0");
    size_t need = 0;
    spork_confidence_workspace_bytes(n_rows, vocab, &need);
    if (ws_bytes < need) return fail(SPORK_E_CAPACITY, "workspace too small");
    if (need > 0 && (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0))
      return fail(SPORK_E_INVAL, "workspace must be non-NULL and 256-byte aligned");
    spork::ConfArgs a{};
    a.logits = logits;
    a.logits_dtype = logits_dtype;
    a.vocab = vocab;
    a.n_rows = n_rows;
    a.chunks = spork::accept_chunks(n_rows, vocab);
    a.n_probes = n_probes;
    a.span_off = span_off;
    a.theta = theta;
    a.argmax_out = argmax_out;
    a.logprob_out = logprob_out;
    a.confidence_out = confidence_out;
    a.commit_out = commit_out;
    const size_t units = static_cast<size_t>(n_rows) * a.chunks;
    a.keys = static_cast<uint64_t*>(workspace);
    a.ms = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + units * sizeof(uint64_t));
    const int rc = hip_status(
        timed(SPORK_KERNEL_CONF_CHUNKS, stream, [&] { return spork::launch_conf_chunks(a, stream); }),
        "spork_probe_confidence (chunks)");
    if (rc != SPORK_OK) return rc;
    return hip_status(timed(SPORK_KERNEL_CONF_FINAL, stream, [&] { return spork::launch_conf_final(a, stream); }),
                      "spork_probe_confidence (final)");
  });
}

int spork_ngram_workspace_bytes(int32_t n_seqs, int64_t max_len, size_t* bytes) {
  if (bytes == nullptr) return fail(SPORK_E_INVAL, "bytes is NULL");
  if (n_seqs < 0 || max_len < 0 || max_len > INT32_MAX)
    return fail(SPORK_E_INVAL, "n_seqs >= 0 and 0 <= max_len < 2^31 required");
  *bytes = static_cast<size_t>(n_seqs) * spork::ngram_chunks(max_len) * sizeof(uint64_t);
  return SPORK_OK;
}

int spork_ngram_propose(const int32_t* tokens, const int64_t* seq_off, int32_t n_seqs, int64_t max_len,
                        int32_t n_min, int32_t n_max, int32_t k, int32_t* drafts, int32_t* n_drafts,
                        void* workspace, size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    if (n_seqs < 0 || max_len < 0 || max_len > INT32_MAX)
      return fail(SPORK_E_INVAL, "n_seqs >= 0 and 0 <= max_len < 2^31 required");
    if (n_min < 1 || n_max < n_min || n_max > spork::kNgramMaxN || k < 0 || k > 4096)
      return fail(SPORK_E_INVAL, "1 <= n_min <= n_max <= 32 and 0 <= k <= 4096 required");
    if (n_seqs > 0 && (tokens == nullptr || seq_off == nullptr || n_drafts == nullptr || (k > 0 && drafts == nullptr)))
      return fail(SPORK_E_INVAL, "NULL pointer");
    size_t need = 0;
    spork_ngram_workspace_bytes(n_seqs, max_len, &need);
    if (ws_bytes < need) return fail(SPORK_E_CAPACITY, "workspace too small");
    if (need > 0 && (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0))
      return fail(SPORK_E_INVAL, "workspace must be non-NULL and 256-byte aligned");
    if (static_cast<int64_t>(n_seqs) * spork::ngram_chunks(max_len) > INT32_MAX)
      return fail(SPORK_E_INVAL, "batch too large");
    spork::NgramArgs a{};
    a.tokens = tokens;
    a.seq_off = seq_off;
    a.n_seqs = n_seqs;
    a.n_chunks = spork::ngram_chunks(max_len);
    a.n_min = n_min;
    a.n_max = n_max;
    a.k = k;
    a.keys = static_cast<uint64_t*>(workspace);
    a.drafts = drafts;
    a.n_drafts = n_drafts;
    const int rc = hip_status(
        timed(SPORK_KERNEL_NGRAM_SCAN, stream, [&] { return spork::launch_ngram_scan(a, stream); }),
        "spork_ngram_propose (scan)");
    if (rc != SPORK_OK) return rc;
    return hip_status(timed(SPORK_KERNEL_NGRAM_DRAFTS, stream, [&] { return spork::launch_ngram_drafts(a, stream); }),
                      "spork_ngram_propose (drafts)");
  });
}

int spork_read_ceiling(const void* src, int64_t bytes, int32_t grid, int32_t mode, uint32_t* sink,
                       hipStream_t stream) {
  return guarded([&] {
    if (src == nullptr || sink == nullptr) return fail(SPORK_E_INVAL, "NULL pointer");
    if (!aligned16(src) || bytes <= 0 || bytes % 16 != 0) return fail(SPORK_E_INVAL, "src 16-byte aligned, bytes a positive multiple of 16");
    if (grid < 1 || grid > 65536 || mode < 0 || mode > 3) return fail(SPORK_E_INVAL, "1 <= grid <= 65536 and mode 0 to 3");
    if ((mode == 1 || mode == 3) && bytes % (static_cast<int64_t>(grid) * 16384) != 0)
      return fail(SPORK_E_INVAL, "mode 1: bytes must be a multiple of grid * 16384");
    return hip_status(timed(SPORK_KERNEL_READ_CEILING, stream,
                            [&] { return spork::launch_read_ceiling(src, bytes, grid, mode, sink, stream); }),
                      "spork_read_ceiling");
  });
}

int spork_timing_enable(int32_t on) {
  g_timing.on = on != 0;
  return SPORK_OK;
}

int spork_timing_read(float* ms_out, int32_t* launches_out) {
  if (ms_out == nullptr) return fail(SPORK_E_INVAL, "ms_out is NULL");
  for (int k = 0; k < SPORK_KERNEL_KINDS; ++k) {
    ms_out[k] = 0.0f;
    if (launches_out) launches_out[k] = 0;
  }
  int rc = SPORK_OK;
  for (const auto& m : g_timing.marks) {
    hipEvent_t b = g_timing.pool[m.second], e = g_timing.pool[m.second + 1];
    float ms = 0.0f;
    if (hipEventSynchronize(e) != hipSuccess || hipEventElapsedTime(&ms, b, e) != hipSuccess) {
      rc = fail(SPORK_E_HIP, "spork_timing_read: event not readable");
      continue;
    }
    ms_out[m.first] += ms;
    if (launches_out) launches_out[m.first] += 1;
  }
  g_timing.marks.clear();
  g_timing.used = 0;
  return rc;
}

}  // extern "C"
