// Host side of the SCD codec's C ABI: argument validation, routing, job tables and launches.
//
// Every entry point validates all of its arguments before the first launch, so a non-OK status
// other than SCD_ERR_HIP means nothing ran.  No entry point allocates device memory, synchronises
// or keeps state beyond the thread-local text of the last error; the streamed decode creates (and
// releases) the events that order its copies and launches.
#include "../../include/scd.h"

#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "scd_kernels.h"

namespace {

thread_local std::string g_last_error;

scd_status_t fail(scd_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

scd_status_t ok() {
  g_last_error.clear();
  return SCD_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

scd_status_t check_model(const scd_model_t* m) {
  if (m == nullptr) return fail(SCD_ERR_NULL, "model is NULL");
  if (m->is_patch == nullptr || m->rank_k == nullptr || m->rank_v == nullptr ||
      m->rank_h == nullptr)
    return fail(SCD_ERR_NULL, "model routing or rank arrays are NULL");
  if (m->n_layers < 1) return fail(SCD_ERR_SHAPE, "n_layers must be >= 1 (got %d)", m->n_layers);
  if (m->n_kv_heads < 1) return fail(SCD_ERR_SHAPE, "n_kv_heads must be >= 1 (got %d)", m->n_kv_heads);
  if (m->head_dim <= 0 || (m->head_dim & 1))
    return fail(SCD_ERR_SHAPE, "head_dim must be positive and even (got %d)", m->head_dim);
  if (m->head_dim != 32 && m->head_dim != 64 && m->head_dim != 128)
    return fail(SCD_ERR_UNSUPPORTED, "head_dim %d unsupported (32, 64 or 128)", m->head_dim);
  const int64_t D = static_cast<int64_t>(m->n_kv_heads) * m->head_dim;
  if (m->basis_width <= 0 || m->basis_width % m->head_dim != 0 || D % m->basis_width != 0)
    return fail(SCD_ERR_SHAPE,
                "basis_width %d must be a multiple of head_dim %d that divides D = %lld",
                m->basis_width, m->head_dim, static_cast<long long>(D));
  if (m->d_model <= 0 || m->d_model % 32 != 0)
    return fail(SCD_ERR_UNSUPPORTED, "d_model %d must be a positive multiple of 32", m->d_model);
  if (m->dtype != SCD_F32 && m->dtype != SCD_BF16)
    return fail(SCD_ERR_SHAPE, "dtype %d unknown", m->dtype);
  if (!(m->rope_theta > 1.0)) return fail(SCD_ERR_SHAPE, "rope_theta must be > 1");
  return SCD_OK;
}

scd_status_t check_rank(const char* what, int layer, int32_t r, int32_t hi) {
  if (r < 16 || r % 16 != 0 || r > hi)
    return fail(SCD_ERR_SCHEDULE, "%s of layer %d is %d; must be a multiple of 16 in [16, %d]",
                what, layer, r, hi);
  return SCD_OK;
}

scd_status_t check_batch(const scd_batch_t* b) {
  if (b == nullptr) return fail(SCD_ERR_NULL, "batch is NULL");
  if (b->n_seqs < 1) return fail(SCD_ERR_SHAPE, "n_seqs must be >= 1 (got %d)", b->n_seqs);
  if (b->n_tokens < 0) return fail(SCD_ERR_SHAPE, "n_tokens must be >= 0");
  if (b->n_tokens > (int64_t{1} << 31) - 1)
    return fail(SCD_ERR_UNSUPPORTED, "n_tokens above 2^31 - 1");
  if (b->cu_seqlens == nullptr && b->n_seqs != 1)
    return fail(SCD_ERR_NULL, "cu_seqlens is NULL but n_seqs = %d", b->n_seqs);
  return SCD_OK;
}

scd_status_t check_rope(const void* table, int64_t max_position) {
  if (table == nullptr) return fail(SCD_ERR_WORKSPACE, "RoPE table is NULL");
  if (!aligned16(table)) return fail(SCD_ERR_ALIGN, "RoPE table is not 16-byte aligned");
  if (max_position < 1) return fail(SCD_ERR_WORKSPACE, "max_position must be >= 1");
  return SCD_OK;
}

// A required per-layer device pointer: the array and its entry must be non-NULL and aligned.
scd_status_t need_ptr(const void* const* arr, int layer, const char* name) {
  if (arr == nullptr) return fail(SCD_ERR_NULL, "%s array is NULL", name);
  if (arr[layer] == nullptr) return fail(SCD_ERR_NULL, "%s[%d] is NULL", name, layer);
  if (!aligned16(arr[layer]))
    return fail(SCD_ERR_ALIGN, "%s[%d] is not 16-byte aligned", name, layer);
  return SCD_OK;
}

// A per-layer buffer sized by the token count: it may be NULL when the batch has no tokens.
scd_status_t need_tok_ptr(const void* const* arr, int layer, const char* name, int64_t n_tokens) {
  if (n_tokens == 0 && (arr == nullptr || arr[layer] == nullptr)) return SCD_OK;
  return need_ptr(arr, layer, name);
}

// An optional per-layer device pointer: NULL array or NULL entry means absent.
scd_status_t opt_ptr(const void* const* arr, int layer, const char* name, const void** out) {
  *out = (arr == nullptr) ? nullptr : arr[layer];
  if (*out != nullptr && !aligned16(*out))
    return fail(SCD_ERR_ALIGN, "%s[%d] is not 16-byte aligned", name, layer);
  return SCD_OK;
}

#define SCD_TRY(expr)                  \
  do {                                 \
    const scd_status_t s_ = (expr);    \
    if (s_ != SCD_OK) return s_;       \
  } while (0)

// Packs jobs into launches of at most kMaxJobs jobs each.
class JobPacker {
 public:
  JobPacker(const scd::GemmParams& base, int bm, int bn) : base_(base), bm_(bm), bn_(bn) {}
  void add(const scd::GemmJob& j) { jobs_.push_back(j); }
  std::vector<scd::GemmParams> build() const {
    std::vector<scd::GemmParams> out;
    const int64_t mt = (base_.m + bm_ - 1) / bm_;
    for (size_t s = 0; s < jobs_.size(); s += scd::kMaxJobs) {
      scd::GemmParams p = base_;
      p.n_jobs = 0;
      int64_t tiles = 0;
      for (size_t i = s; i < jobs_.size() && i < s + scd::kMaxJobs; ++i) {
        scd::GemmJob j = jobs_[i];
        j.tile_begin = static_cast<int32_t>(tiles);
        tiles += mt * ((j.n + bn_ - 1) / bn_);
        p.jobs[p.n_jobs++] = j;
      }
      p.total_tiles = static_cast<int32_t>(tiles);
      out.push_back(p);
    }
    return out;
  }

 private:
  scd::GemmParams base_;
  int bm_, bn_;
  std::vector<scd::GemmJob> jobs_;
};

scd::GemmParams base_params(const scd_model_t* m, const scd_batch_t* b, int64_t rows, int g,
                            const void* rope, int64_t max_pos) {
  scd::GemmParams p{};
  p.n_jobs = 0;
  p.total_tiles = 0;
  p.m = rows;
  p.g = g;
  p.head_dim = m->head_dim;
  p.n_seqs = b->n_seqs;
  p.cu_seqlens = b->cu_seqlens;
  p.pos0 = b->pos0;
  p.rope = static_cast<const float2*>(rope);
  p.max_pos = max_pos;
  return p;
}

scd_status_t run(scd::Op op, const std::vector<scd::GemmParams>& launches, int dtype,
                 hipStream_t stream) {
  for (const auto& p : launches) {
    const hipError_t e = scd::launch_gemm(op, dtype == SCD_BF16, p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

// Splits jobs into launches of equal key (one kernel instance each), in first-seen order.
template <typename KeyFn>
std::vector<std::vector<scd::GemmJob>> group_by(const std::vector<scd::GemmJob>& jobs, KeyFn key) {
  std::vector<std::vector<scd::GemmJob>> groups;
  std::vector<int> keys;
  for (const auto& j : jobs) {
    const int k = key(j);
    size_t g = 0;
    while (g < keys.size() && keys[g] != k) ++g;
    if (g == keys.size()) {
      keys.push_back(k);
      groups.emplace_back();
    }
    groups[g].push_back(j);
  }
  return groups;
}

template <typename LaunchFn>
scd_status_t run_groups(const scd::GemmParams& base, int bm, int bn,
                        const std::vector<std::vector<scd::GemmJob>>& groups, LaunchFn launch,
                        const char* what) {
  for (const auto& g : groups) {
    JobPacker jp(base, bm, bn);
    for (const auto& j : g) jp.add(j);
    for (const auto& p : jp.build()) {
      const hipError_t e = launch(p);
      if (e != hipSuccess)
        return fail(SCD_ERR_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
    }
  }
  return ok();
}

int64_t kv_width(const scd_model_t* m) {
  return static_cast<int64_t>(m->n_kv_heads) * m->head_dim;
}

}  // namespace

extern "C" {

int32_t scd_abi_version(void) { return 5; }

const char* scd_status_string(scd_status_t s) {
  switch (s) {
    case SCD_OK: return "ok";
    case SCD_ERR_NULL: return "null pointer";
    case SCD_ERR_SHAPE: return "invalid shape";
    case SCD_ERR_SCHEDULE: return "invalid schedule or rank";
    case SCD_ERR_ALIGN: return "misaligned pointer";
    case SCD_ERR_UNSUPPORTED: return "unsupported configuration";
    case SCD_ERR_WORKSPACE: return "missing or invalid RoPE table";
    case SCD_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* scd_last_error(void) { return g_last_error.c_str(); }

// Rows a RoPE table for max_position holds (never fewer than kRopeMinRows).
static int64_t rope_rows(int64_t max_position) {
  return max_position > scd::kRopeMinRows ? max_position : scd::kRopeMinRows;
}

size_t scd_rope_table_bytes(const scd_model_t* model, int64_t max_position) {
  if (model == nullptr || model->head_dim <= 0 || max_position < 1) return 0;
  return static_cast<size_t>(rope_rows(max_position)) * static_cast<size_t>(model->head_dim / 2) *
         sizeof(float2);
}

scd_status_t scd_rope_table(const scd_model_t* model, int64_t max_position, void* table,
                            size_t table_bytes, hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_rope(table, max_position));
  if (table_bytes < scd_rope_table_bytes(model, max_position))
    return fail(SCD_ERR_WORKSPACE, "table_bytes %zu < %zu needed", table_bytes,
                scd_rope_table_bytes(model, max_position));
  if (max_position > (int64_t{1} << 31))
    return fail(SCD_ERR_UNSUPPORTED, "max_position above 2^31");
  const hipError_t e = scd::launch_rope_table(static_cast<float2*>(table), rope_rows(max_position),
                                              model->head_dim, model->rope_theta, stream);
  if (e != hipSuccess) return fail(SCD_ERR_HIP, "rope table launch failed: %s", hipGetErrorString(e));
  return ok();
}

scd_status_t scd_positions(const scd_batch_t* batch, int32_t* pos_out, hipStream_t stream) {
  SCD_TRY(check_batch(batch));
  if (batch->n_tokens == 0) return ok();
  if (pos_out == nullptr) return fail(SCD_ERR_NULL, "pos_out is NULL");
  const hipError_t e = scd::launch_positions(pos_out, batch->n_tokens, batch->n_seqs,
                                             batch->cu_seqlens, batch->pos0, stream);
  if (e != hipSuccess) return fail(SCD_ERR_HIP, "positions launch failed: %s", hipGetErrorString(e));
  return ok();
}

scd_status_t scd_schedule(const scd_model_t* model, int32_t* reuse_layers, int32_t* n_reuse,
                          int32_t* patch_layers, int32_t* n_patch) {
  if (model == nullptr || model->is_patch == nullptr) return fail(SCD_ERR_NULL, "model is NULL");
  if (model->n_layers < 1) return fail(SCD_ERR_SHAPE, "n_layers must be >= 1");
  if (n_reuse == nullptr || n_patch == nullptr) return fail(SCD_ERR_NULL, "count outputs are NULL");
  int32_t nr = 0, np = 0;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) {
      if (patch_layers != nullptr) patch_layers[np] = l;
      ++np;
    } else {
      if (reuse_layers != nullptr) reuse_layers[nr] = l;
      ++nr;
    }
  }
  *n_reuse = nr;
  *n_patch = np;
  return ok();
}

size_t scd_payload_bytes(const scd_model_t* model, int64_t n_tokens, int64_t* offsets) {
  if (check_model(model) != SCD_OK || n_tokens < 0) return 0;
  const int64_t g = kv_width(model) / model->basis_width;
  const int64_t eb = model->dtype == SCD_BF16 ? 2 : 4;
  int64_t total = 0;
  if (offsets != nullptr) offsets[0] = 0;
  for (int l = 0; l < model->n_layers; ++l) {
    const int64_t n = model->is_patch[l]
                          ? n_tokens * model->rank_h[l]
                          : n_tokens * g * (int64_t{model->rank_k[l]} + model->rank_v[l]);
    total += n * eb;
    if (offsets != nullptr) offsets[l + 1] = total;
  }
  return static_cast<size_t>(total);
}

scd_status_t scd_encode(const scd_model_t* model, const scd_batch_t* batch,
                        const void* rope_table, int64_t max_position,
                        const void* const* k_in, const void* const* v_in,
                        const void* const* h_in,
                        const void* const* w_enc_k, const void* const* w_enc_v,
                        const void* const* w_enc_h,
                        const void* const* mu_k, const void* const* mu_v,
                        void* const* z_k, void* const* z_v, void* const* z_h,
                        hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  const int w = model->basis_width;
  const int g = static_cast<int>(kv_width(model) / w);
  const int rk_max = w < 256 ? w : 256;
  const int rh_max = model->d_model < 256 ? model->d_model : 256;
  bool any_reuse = false;
  for (int l = 0; l < model->n_layers; ++l) {
    const void* tmp;
    if (model->is_patch[l]) {
      SCD_TRY(check_rank("rank_h", l, model->rank_h[l], rh_max));
      SCD_TRY(need_tok_ptr(h_in, l, "h_in", batch->n_tokens));
      SCD_TRY(need_ptr(w_enc_h, l, "w_enc_h"));
      SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(z_h), l, "z_h", batch->n_tokens));
    } else {
      any_reuse = true;
      SCD_TRY(check_rank("rank_k", l, model->rank_k[l], rk_max));
      SCD_TRY(check_rank("rank_v", l, model->rank_v[l], rk_max));
      SCD_TRY(need_tok_ptr(k_in, l, "k_in", batch->n_tokens));
      SCD_TRY(need_tok_ptr(v_in, l, "v_in", batch->n_tokens));
      SCD_TRY(need_ptr(w_enc_k, l, "w_enc_k"));
      SCD_TRY(need_ptr(w_enc_v, l, "w_enc_v"));
      SCD_TRY(opt_ptr(mu_k, l, "mu_k", &tmp));
      SCD_TRY(opt_ptr(mu_v, l, "mu_v", &tmp));
      SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(z_k), l, "z_k", batch->n_tokens));
      SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(z_v), l, "z_v", batch->n_tokens));
    }
  }
  if (any_reuse && batch->n_tokens > 0) SCD_TRY(check_rope(rope_table, max_position));
  if (batch->n_tokens == 0) return ok();

  const int64_t T = batch->n_tokens;
  const bool bf16 = model->dtype == SCD_BF16;
  const bool hd_ok = model->head_dim == 64 || model->head_dim == 128;
  const bool fast_kv = bf16 && hd_ok && w % 128 == 0;
  const bool fast_h = bf16 && model->d_model % 128 == 0;
  std::vector<scd::GemmJob> kv_jobs, h_jobs;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) {
      h_jobs.push_back({h_in[l], w_enc_h[l], z_h[l], nullptr, model->rank_h[l], model->d_model, 0, 0});
    } else {
      const void* mk = mu_k ? mu_k[l] : nullptr;
      const void* mv = mu_v ? mu_v[l] : nullptr;
      kv_jobs.push_back({k_in[l], w_enc_k[l], z_k[l], mk, model->rank_k[l], w,
                         scd::kDeropeIn | scd::kVecIn, 0});
      kv_jobs.push_back({v_in[l], w_enc_v[l], z_v[l], mv, model->rank_v[l], w, scd::kVecIn, 0});
    }
  }
  const scd::GemmParams kv_base = base_params(model, batch, T * g, g, rope_table, max_position);
  const scd::GemmParams h_base = base_params(model, batch, T, 1, rope_table, max_position);
  // one launch per (rank, branch kind, offset present): each is its own kernel instance
  auto by_kind = [](const scd::GemmJob& j) {
    const bool mu = (j.flags & scd::kVecIn) != 0 && j.vec != nullptr;
    return j.n * 4 + ((j.flags & scd::kDeropeIn) != 0 ? 2 : 0) + (mu ? 1 : 0);
  };
  auto enc = [&](const scd::GemmParams& p) { return scd::launch_encode_bf16(p, stream); };
  if (fast_kv) {
    // tiles of 128 code columns: a rank above 128 takes two workgroups per row tile
    SCD_TRY(run_groups(kv_base, scd::kEncodeRows, 128, group_by(kv_jobs, by_kind), enc, "encode"));
  } else {
    JobPacker jp(kv_base, scd::kGenericBM, scd::kGenericBN);
    for (const auto& j : kv_jobs) jp.add(j);
    SCD_TRY(run(scd::Op::kEncodeKV, jp.build(), model->dtype, stream));
  }
  if (fast_h)
    return run_groups(h_base, scd::kEncodeRows, 128, group_by(h_jobs, by_kind), enc, "encode");
  JobPacker hp(h_base, scd::kGenericBM, scd::kGenericBN);
  for (const auto& j : h_jobs) hp.add(j);
  return run(scd::Op::kEncodeH, hp.build(), model->dtype, stream);
}

namespace {

// Validation half of the Reuse decode; *any is set when the model has a Reuse layer.
scd_status_t check_reuse_decode(const scd_model_t* model, const scd_batch_t* batch,
                                const void* rope_table, int64_t max_position,
                                const void* const* z_k, const void* const* z_v,
                                const void* const* w_dec_k, const void* const* w_dec_v,
                                const void* const* mu_k, const void* const* mu_v,
                                void* const* k_cache, void* const* v_cache, bool* any_out) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  const int w = model->basis_width;
  const int rk_max = w < 256 ? w : 256;
  bool any = false;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) continue;
    any = true;
    const void* tmp;
    SCD_TRY(check_rank("rank_k", l, model->rank_k[l], rk_max));
    SCD_TRY(check_rank("rank_v", l, model->rank_v[l], rk_max));
    SCD_TRY(need_tok_ptr(z_k, l, "z_k", batch->n_tokens));
    SCD_TRY(need_tok_ptr(z_v, l, "z_v", batch->n_tokens));
    SCD_TRY(need_ptr(w_dec_k, l, "w_dec_k"));
    SCD_TRY(need_ptr(w_dec_v, l, "w_dec_v"));
    SCD_TRY(opt_ptr(mu_k, l, "mu_k", &tmp));
    SCD_TRY(opt_ptr(mu_v, l, "mu_v", &tmp));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(k_cache), l, "k_cache", batch->n_tokens));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(v_cache), l, "v_cache", batch->n_tokens));
  }
  if (any && batch->n_tokens > 0) SCD_TRY(check_rope(rope_table, max_position));
  *any_out = any;
  return SCD_OK;
}

// Launch half of the Reuse decode, on arguments check_reuse_decode accepted.
scd_status_t enqueue_reuse_decode(const scd_model_t* model, const scd_batch_t* batch,
                                  const void* rope_table, int64_t max_position,
                                  const void* const* z_k, const void* const* z_v,
                                  const void* const* w_dec_k, const void* const* w_dec_v,
                                  const void* const* mu_k, const void* const* mu_v,
                                  void* const* k_cache, void* const* v_cache,
                                  hipStream_t stream) {
  const int w = model->basis_width;
  const int g = static_cast<int>(kv_width(model) / w);
  const int64_t T = batch->n_tokens;
  bool fast = model->dtype == SCD_BF16 && (model->head_dim == 64 || model->head_dim == 128) &&
              w % 128 == 0 && batch->n_seqs <= scd::kMaxLdsSeqs;
  std::vector<scd::GemmJob> jobs;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) continue;
    const void* mk = mu_k ? mu_k[l] : nullptr;
    const void* mv = mu_v ? mu_v[l] : nullptr;
    jobs.push_back({z_k[l], w_dec_k[l], k_cache[l], mk, w, model->rank_k[l],
                    scd::kRopeOut | scd::kVecOut, 0});
    jobs.push_back({z_v[l], w_dec_v[l], v_cache[l], mv, w, model->rank_v[l], scd::kVecOut, 0});
    if (model->rank_k[l] % 32 != 0 || model->rank_v[l] % 32 != 0) fast = false;
  }
  const scd::GemmParams base = base_params(model, batch, T * g, g, rope_table, max_position);
  if (!fast) {
    JobPacker jp(base, scd::kGenericBM, scd::kGenericBN);
    for (const auto& j : jobs) jp.add(j);
    return run(scd::Op::kReuseDecode, jp.build(), model->dtype, stream);
  }
  // one launch per (rank, branch): key and value jobs run different kernel instances
  for (const auto& grp : group_by(jobs, [](const scd::GemmJob& j) {
         return j.k * 2 + ((j.flags & scd::kRopeOut) != 0 ? 1 : 0);
       })) {
    const int nhg = scd::decode_channel_groups(grp[0].k, w);
    scd::GemmParams gp = base;
    JobPacker jp(gp, scd::decode_tile_rows(nhg, grp[0].k), 128 * nhg);
    for (const auto& j : grp) jp.add(j);
    for (const auto& lp : jp.build()) {
      const hipError_t e = scd::launch_decode_bf16(nhg, lp, stream);
      if (e != hipSuccess)
        return fail(SCD_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
    }
  }
  return SCD_OK;
}

}  // namespace

scd_status_t scd_reuse_decode(const scd_model_t* model, const scd_batch_t* batch,
                              const void* rope_table, int64_t max_position,
                              const void* const* z_k, const void* const* z_v,
                              const void* const* w_dec_k, const void* const* w_dec_v,
                              const void* const* mu_k, const void* const* mu_v,
                              void* const* k_cache, void* const* v_cache, hipStream_t stream) {
  bool any = false;
  SCD_TRY(check_reuse_decode(model, batch, rope_table, max_position, z_k, z_v, w_dec_k, w_dec_v,
                             mu_k, mu_v, k_cache, v_cache, &any));
  if (!any || batch->n_tokens == 0) return ok();
  SCD_TRY(enqueue_reuse_decode(model, batch, rope_table, max_position, z_k, z_v, w_dec_k,
                               w_dec_v, mu_k, mu_v, k_cache, v_cache, stream));
  return ok();
}

scd_status_t scd_payload_views(const scd_model_t* model, int64_t n_tokens, void* payload,
                               void** z_k, void** z_v, void** z_h) {
  SCD_TRY(check_model(model));
  if (n_tokens < 0) return fail(SCD_ERR_SHAPE, "n_tokens must be >= 0");
  if (payload == nullptr) return fail(SCD_ERR_NULL, "payload is NULL");
  if (!aligned16(payload)) return fail(SCD_ERR_ALIGN, "payload is not 16-byte aligned");
  if (z_k == nullptr || z_v == nullptr || z_h == nullptr)
    return fail(SCD_ERR_NULL, "view arrays must not be NULL");
  const int w = model->basis_width;
  const int rk_max = w < 256 ? w : 256;
  const int rh_max = model->d_model < 256 ? model->d_model : 256;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) {
      SCD_TRY(check_rank("rank_h", l, model->rank_h[l], rh_max));
    } else {
      SCD_TRY(check_rank("rank_k", l, model->rank_k[l], rk_max));
      SCD_TRY(check_rank("rank_v", l, model->rank_v[l], rk_max));
    }
  }
  // Ranks are multiples of 16, so every view below inherits the base's 16-byte alignment.
  const int64_t g = kv_width(model) / w;
  const int64_t eb = model->dtype == SCD_BF16 ? 2 : 4;
  char* base = static_cast<char*>(payload);
  int64_t off = 0;
  for (int l = 0; l < model->n_layers; ++l) {
    z_k[l] = z_v[l] = z_h[l] = nullptr;
    if (model->is_patch[l]) {
      z_h[l] = base + off;
      off += n_tokens * model->rank_h[l] * eb;
    } else {
      z_k[l] = base + off;
      off += n_tokens * g * model->rank_k[l] * eb;
      z_v[l] = base + off;
      off += n_tokens * g * model->rank_v[l] * eb;
    }
  }
  return ok();
}

namespace {

// Owns the events of one streamed call; destroying a recorded event is safe (HIP releases it once
// the recorded work completes).
struct EventSet {
  std::vector<hipEvent_t> ev;
  ~EventSet() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
  hipError_t add(hipEvent_t* out) {
    const hipError_t e = hipEventCreateWithFlags(out, hipEventDisableTiming);
    if (e == hipSuccess) ev.push_back(*out);
    return e;
  }
};

}  // namespace

scd_status_t scd_reuse_decode_streamed(const scd_model_t* model, const scd_batch_t* batch,
                                       const void* rope_table, int64_t max_position,
                                       const void* payload_src, void* payload_dst,
                                       int32_t layers_per_group,
                                       const void* const* w_dec_k, const void* const* w_dec_v,
                                       const void* const* mu_k, const void* const* mu_v,
                                       void* const* k_cache, void* const* v_cache,
                                       hipStream_t copy_stream, hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  if (layers_per_group < 1)
    return fail(SCD_ERR_SHAPE, "layers_per_group must be >= 1 (got %d)", layers_per_group);
  const int L = model->n_layers;
  const int64_t T = batch->n_tokens;
  std::vector<int64_t> offs(L + 1);
  const size_t total = scd_payload_bytes(model, T, offs.data());
  std::vector<void*> zk(L, nullptr), zv(L, nullptr), zh(L, nullptr);
  if (total > 0) {  // an empty payload (no tokens) may come with NULL buffers
    if (payload_src == nullptr) return fail(SCD_ERR_NULL, "payload_src is NULL");
    if (payload_dst == nullptr) return fail(SCD_ERR_NULL, "payload_dst is NULL");
    SCD_TRY(scd_payload_views(model, T, payload_dst, zk.data(), zv.data(), zh.data()));
  }
  bool any = false;
  SCD_TRY(check_reuse_decode(model, batch, rope_table, max_position, zk.data(), zv.data(),
                             w_dec_k, w_dec_v, mu_k, mu_v, k_cache, v_cache, &any));
  if (total == 0) return ok();

  auto hip_fail = [](const char* what, hipError_t e) {
    return fail(SCD_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
  };
  EventSet events;
  hipEvent_t ready;  // work already queued on stream (producer of payload_src, readers of dst)
  hipError_t e = events.add(&ready);
  if (e != hipSuccess) return hip_fail("event creation", e);
  if ((e = hipEventRecord(ready, stream)) != hipSuccess) return hip_fail("event record", e);
  if ((e = hipStreamWaitEvent(copy_stream, ready, 0)) != hipSuccess)
    return hip_fail("stream wait", e);

  const char* src = static_cast<const char*>(payload_src);
  char* dst = static_cast<char*>(payload_dst);
  for (int l0 = 0; l0 < L; l0 += layers_per_group) {
    const int l1 = l0 + layers_per_group < L ? l0 + layers_per_group : L;
    const int64_t bytes = offs[l1] - offs[l0];
    if (bytes == 0) continue;
    if ((e = hipMemcpyAsync(dst + offs[l0], src + offs[l0], static_cast<size_t>(bytes),
                            hipMemcpyDefault, copy_stream)) != hipSuccess)
      return hip_fail("payload copy", e);
    hipEvent_t landed;
    if ((e = events.add(&landed)) != hipSuccess) return hip_fail("event creation", e);
    if ((e = hipEventRecord(landed, copy_stream)) != hipSuccess) return hip_fail("event record", e);
    if ((e = hipStreamWaitEvent(stream, landed, 0)) != hipSuccess)
      return hip_fail("stream wait", e);
    if (!any || T == 0) continue;
    // the group's layers as a model of their own: routing and rank arrays start at l0
    scd_model_t sub = *model;
    sub.n_layers = l1 - l0;
    sub.is_patch += l0;
    sub.rank_k += l0;
    sub.rank_v += l0;
    sub.rank_h += l0;
    bool sub_any = false;
    for (int l = l0; l < l1; ++l) sub_any = sub_any || !model->is_patch[l];
    if (!sub_any) continue;
    SCD_TRY(enqueue_reuse_decode(&sub, batch, rope_table, max_position, zk.data() + l0,
                                 zv.data() + l0, w_dec_k + l0, w_dec_v + l0,
                                 mu_k ? mu_k + l0 : nullptr, mu_v ? mu_v + l0 : nullptr,
                                 k_cache + l0, v_cache + l0, stream));
  }
  return ok();
}

}  // extern "C"

namespace {

// The aligner's first product act = SiLU(z_h w1^T + b1) for `jobs` (one per Patch layer, K = r_H).
// It is a short contraction whose time is writing act: the shape of a Reuse decode (code x basis
// + offset), so the bf16 decode kernel takes every job it can (r_H % 32 == 0, r_H <= 256), one
// launch per rank; the other jobs take the bf16 GEMM body when `fast` (r_H % 64 == 0 and
// hidden % 128 == 0), else the generic kernel.
scd_status_t enqueue_align_first(const scd_model_t* model, const scd_batch_t* batch, int hidden,
                                 const std::vector<scd::GemmJob>& jobs, bool fast,
                                 hipStream_t stream) {
  const scd::GemmParams base = base_params(model, batch, batch->n_tokens, 1, nullptr, 0);
  const bool decode_ok = model->dtype == SCD_BF16 && hidden % 128 == 0 &&
                         (model->head_dim == 64 || model->head_dim == 128) &&
                         batch->n_seqs <= scd::kMaxLdsSeqs;
  std::vector<scd::GemmJob> on_decode, rest;
  for (const auto& j : jobs)
    (decode_ok && j.k % 32 == 0 && j.k <= 256 ? on_decode : rest).push_back(j);
  for (const auto& grp : group_by(on_decode, [](const scd::GemmJob& j) { return j.k; })) {
    const int nhg = scd::decode_channel_groups(grp[0].k, hidden);
    JobPacker jp(base, scd::decode_tile_rows(nhg, grp[0].k), 128 * nhg);
    for (const auto& j : grp) jp.add(j);
    for (const auto& lp : jp.build()) {
      const hipError_t e = scd::launch_decode_bf16(nhg, lp, stream, true);
      if (e != hipSuccess)
        return fail(SCD_ERR_HIP, "aligner launch failed: %s", hipGetErrorString(e));
    }
  }
  if (rest.empty()) return ok();
  bool gemm_ok = fast;
  for (const auto& j : rest)
    if (j.k % 64 != 0) gemm_ok = false;
  JobPacker jp(base, gemm_ok ? scd::kPatchBM : scd::kGenericBM,
               gemm_ok ? scd::kPatchBN : scd::kGenericBN);
  for (const auto& j : rest) jp.add(j);
  if (!gemm_ok) return run(scd::Op::kPatchAlign, jp.build(), model->dtype, stream);
  for (const auto& p : jp.build()) {
    const hipError_t e = scd::launch_align_bf16(p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "aligner launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

}  // namespace

extern "C" {

scd_status_t scd_patch_kv(const scd_model_t* model, const scd_batch_t* batch,
                          const void* rope_table, int64_t max_position,
                          const void* const* h_hat,
                          const void* const* w_k, const void* const* w_v,
                          const void* const* b_k, const void* const* b_v,
                          void* const* k_cache, void* const* v_cache, hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  bool any = false;
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    any = true;
    const void* tmp;
    SCD_TRY(need_tok_ptr(h_hat, l, "h_hat", batch->n_tokens));
    SCD_TRY(need_ptr(w_k, l, "w_k"));
    SCD_TRY(need_ptr(w_v, l, "w_v"));
    SCD_TRY(opt_ptr(b_k, l, "b_k", &tmp));
    SCD_TRY(opt_ptr(b_v, l, "b_v", &tmp));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(k_cache), l, "k_cache", batch->n_tokens));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(v_cache), l, "v_cache", batch->n_tokens));
  }
  if (any && batch->n_tokens > 0) SCD_TRY(check_rope(rope_table, max_position));
  if (!any || batch->n_tokens == 0) return ok();

  const int64_t T = batch->n_tokens;
  const int D = static_cast<int>(kv_width(model));
  const bool fast = model->dtype == SCD_BF16 && model->d_model % 64 == 0 &&
                    (model->head_dim == 64 || model->head_dim == 128) && D % 128 == 0;
  JobPacker jp(base_params(model, batch, T, 1, rope_table, max_position),
               fast ? scd::kPatchBM : scd::kGenericBM, fast ? scd::kPatchBN : scd::kGenericBN);
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    const void* bk = b_k ? b_k[l] : nullptr;
    const void* bv = b_v ? b_v[l] : nullptr;
    jp.add({h_hat[l], w_k[l], k_cache[l], bk, D, model->d_model, scd::kRopeOut | scd::kVecOut, 0});
    jp.add({h_hat[l], w_v[l], v_cache[l], bv, D, model->d_model, scd::kVecOut, 0});
  }
  if (!fast) return run(scd::Op::kPatchKV, jp.build(), model->dtype, stream);
  for (const auto& p : jp.build()) {
    const hipError_t e = scd::launch_patch_bf16(p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "patch launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

scd_status_t scd_patch_align(const scd_model_t* model, const scd_batch_t* batch, int32_t hidden,
                             const void* const* z_h,
                             const void* const* w1, const void* const* b1,
                             const void* const* w2, const void* const* b2,
                             void* const* act, void* const* h_hat, hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  if (hidden < 16 || hidden % 16 != 0)
    return fail(SCD_ERR_SHAPE, "aligner width %d must be a positive multiple of 16", hidden);
  if (model->d_model % 16 != 0)
    return fail(SCD_ERR_SHAPE, "d_model %d must be a multiple of 16 for the aligner",
                model->d_model);
  const int rh_max = model->d_model < 256 ? model->d_model : 256;
  bool any = false;
  // The second product (K = hidden) takes the bf16 GEMM body whenever the widths allow; the first
  // (K = r_H) goes where enqueue_align_first sends it.
  const bool fast2 = model->dtype == SCD_BF16 && hidden % 128 == 0 && model->d_model % 128 == 0;
  std::vector<const void*> acts;
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    any = true;
    const void* tmp;
    SCD_TRY(check_rank("rank_h", l, model->rank_h[l], rh_max));
    SCD_TRY(need_tok_ptr(z_h, l, "z_h", batch->n_tokens));
    SCD_TRY(need_ptr(w1, l, "w1"));
    SCD_TRY(need_ptr(w2, l, "w2"));
    SCD_TRY(opt_ptr(b1, l, "b1", &tmp));
    SCD_TRY(opt_ptr(b2, l, "b2", &tmp));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(act), l, "act", batch->n_tokens));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(h_hat), l, "h_hat",
                         batch->n_tokens));
    if (batch->n_tokens > 0) {
      for (const void* a : acts)
        if (a == act[l])
          return fail(SCD_ERR_SHAPE, "act[%d] repeats an earlier Patch layer's buffer", l);
      acts.push_back(act[l]);
    }
  }
  if (!any || batch->n_tokens == 0) return ok();

  const int64_t T = batch->n_tokens;
  const int d = model->d_model;
  const scd::GemmParams base = base_params(model, batch, T, 1, nullptr, 0);
  // act = SiLU(z_h w1^T + b1) for every Patch layer, then h_hat = act w2^T + b2
  std::vector<scd::GemmJob> first_jobs;
  JobPacker second(base, fast2 ? scd::kPatchBM : scd::kGenericBM,
                   fast2 ? scd::kPatchBN : scd::kGenericBN);
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    first_jobs.push_back({z_h[l], w1[l], act[l], b1 ? b1[l] : nullptr, hidden, model->rank_h[l],
                          scd::kVecOut | scd::kSiluOut, 0});
    second.add({act[l], w2[l], h_hat[l], b2 ? b2[l] : nullptr, d, hidden, scd::kVecOut, 0});
  }
  SCD_TRY(enqueue_align_first(model, batch, hidden, first_jobs,
                              model->dtype == SCD_BF16 && hidden % 128 == 0, stream));
  if (!fast2) return run(scd::Op::kPatchAlign, second.build(), model->dtype, stream);
  for (const auto& p : second.build()) {
    const hipError_t e = scd::launch_align_bf16(p, stream);
    if (e != hipSuccess)
      return fail(SCD_ERR_HIP, "aligner launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

// A per-layer output that must not repeat across the listed layers.
static scd_status_t distinct_layer_outputs(const std::vector<int>& layers, const void* const* arr,
                                           const char* name) {
  for (size_t i = 0; i < layers.size(); ++i)
    for (size_t j = 0; j < i; ++j)
      if (arr[layers[i]] == arr[layers[j]])
        return fail(SCD_ERR_SHAPE, "%s[%d] repeats layer %d's buffer", name, layers[i], layers[j]);
  return SCD_OK;
}

scd_status_t scd_patch_fold(const scd_model_t* model, int32_t hidden,
                            const void* const* w2, const void* const* b2,
                            const void* const* w_k, const void* const* w_v,
                            const void* const* b_k, const void* const* b_v,
                            void* const* w_fold_k, void* const* w_fold_v,
                            void* const* c_k, void* const* c_v, hipStream_t stream) {
  SCD_TRY(check_model(model));
  if (hidden < 16 || hidden % 16 != 0)
    return fail(SCD_ERR_SHAPE, "aligner width %d must be a positive multiple of 16", hidden);
  std::vector<int> layers;
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    layers.push_back(l);
    const void* tmp;
    SCD_TRY(need_ptr(w2, l, "w2"));
    SCD_TRY(opt_ptr(b2, l, "b2", &tmp));
    SCD_TRY(need_ptr(w_k, l, "w_k"));
    SCD_TRY(need_ptr(w_v, l, "w_v"));
    SCD_TRY(opt_ptr(b_k, l, "b_k", &tmp));
    SCD_TRY(opt_ptr(b_v, l, "b_v", &tmp));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(w_fold_k), l, "w_fold_k"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(w_fold_v), l, "w_fold_v"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(c_k), l, "c_k"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(c_v), l, "c_v"));
    if (w_fold_k[l] == w_fold_v[l] || c_k[l] == c_v[l])
      return fail(SCD_ERR_SHAPE, "layer %d's key and value outputs share a buffer", l);
  }
  if (layers.empty()) return ok();
  SCD_TRY(distinct_layer_outputs(layers, reinterpret_cast<const void* const*>(w_fold_k), "w_fold_k"));
  SCD_TRY(distinct_layer_outputs(layers, reinterpret_cast<const void* const*>(w_fold_v), "w_fold_v"));
  SCD_TRY(distinct_layer_outputs(layers, reinterpret_cast<const void* const*>(c_k), "c_k"));
  SCD_TRY(distinct_layer_outputs(layers, reinterpret_cast<const void* const*>(c_v), "c_v"));

  std::vector<scd::FoldJob> jobs;
  for (int l : layers) {
    jobs.push_back({w_k[l], w2[l], b2 ? b2[l] : nullptr, b_k ? b_k[l] : nullptr, w_fold_k[l], c_k[l]});
    jobs.push_back({w_v[l], w2[l], b2 ? b2[l] : nullptr, b_v ? b_v[l] : nullptr, w_fold_v[l], c_v[l]});
  }
  for (size_t done = 0; done < jobs.size(); done += scd::kMaxJobs) {
    scd::FoldParams p{};
    p.n_jobs = 0;
    for (size_t i = done; i < jobs.size() && i < done + scd::kMaxJobs; ++i) p.jobs[p.n_jobs++] = jobs[i];
    p.n = static_cast<int32_t>(kv_width(model));
    p.d_model = model->d_model;
    p.hidden = hidden;
    const hipError_t e = scd::launch_patch_fold(model->dtype == SCD_BF16, p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "fold launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

scd_status_t scd_patch_kv_from_codes(const scd_model_t* model, const scd_batch_t* batch,
                                     const void* rope_table, int64_t max_position, int32_t hidden,
                                     const void* const* z_h,
                                     const void* const* w1, const void* const* b1,
                                     const void* const* w_fold_k, const void* const* w_fold_v,
                                     const void* const* c_k, const void* const* c_v,
                                     void* const* act, void* const* k_cache, void* const* v_cache,
                                     hipStream_t stream) {
  SCD_TRY(check_model(model));
  SCD_TRY(check_batch(batch));
  if (hidden < 16 || hidden % 16 != 0)
    return fail(SCD_ERR_SHAPE, "aligner width %d must be a positive multiple of 16", hidden);
  const int rh_max = model->d_model < 256 ? model->d_model : 256;
  const int64_t T = batch->n_tokens;
  bool any = false;
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    any = true;
    const void* tmp;
    SCD_TRY(check_rank("rank_h", l, model->rank_h[l], rh_max));
    SCD_TRY(need_tok_ptr(z_h, l, "z_h", T));
    SCD_TRY(need_ptr(w1, l, "w1"));
    SCD_TRY(opt_ptr(b1, l, "b1", &tmp));
    SCD_TRY(need_ptr(w_fold_k, l, "w_fold_k"));
    SCD_TRY(need_ptr(w_fold_v, l, "w_fold_v"));
    SCD_TRY(opt_ptr(c_k, l, "c_k", &tmp));
    SCD_TRY(opt_ptr(c_v, l, "c_v", &tmp));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(act), l, "act", T));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(k_cache), l, "k_cache", T));
    SCD_TRY(need_tok_ptr(reinterpret_cast<const void* const*>(v_cache), l, "v_cache", T));
  }
  if (any && T > 0) SCD_TRY(check_rope(rope_table, max_position));
  if (!any || T == 0) return ok();

  const int D = static_cast<int>(kv_width(model));
  const bool fast_first = model->dtype == SCD_BF16 && hidden % 128 == 0;
  const bool fast = model->dtype == SCD_BF16 && hidden % 64 == 0 &&
                    (model->head_dim == 64 || model->head_dim == 128) && D % 128 == 0;
  const scd::GemmParams base = base_params(model, batch, T, 1, rope_table, max_position);
  // Patch layers in order, grouped: a group is a run of consecutive Patch layers whose act buffers
  // are all distinct; each group is one launch of the hidden layer and one of the folded product.
  // A buffer that repeats starts a new group, so a shared act buffer is overwritten only after the
  // product that reads it (stream order).
  std::vector<std::vector<int>> groups;
  for (int l = 0; l < model->n_layers; ++l) {
    if (!model->is_patch[l]) continue;
    bool clash = groups.empty();
    if (!clash)
      for (int m : groups.back())
        if (act[m] == act[l]) clash = true;
    if (clash) groups.emplace_back();
    groups.back().push_back(l);
  }
  for (const auto& grp : groups) {
    std::vector<scd::GemmJob> first;
    JobPacker jp(base, fast ? scd::kPatchBM : scd::kGenericBM, fast ? scd::kPatchBN : scd::kGenericBN);
    for (int l : grp) {
      first.push_back({z_h[l], w1[l], act[l], b1 ? b1[l] : nullptr, hidden, model->rank_h[l],
                       scd::kVecOut | scd::kSiluOut, 0});
      jp.add({act[l], w_fold_k[l], k_cache[l], c_k ? c_k[l] : nullptr, D, hidden,
              scd::kRopeOut | scd::kVecOut, 0});
      jp.add({act[l], w_fold_v[l], v_cache[l], c_v ? c_v[l] : nullptr, D, hidden, scd::kVecOut, 0});
    }
    SCD_TRY(enqueue_align_first(model, batch, hidden, first, fast_first, stream));
    if (!fast) {
      SCD_TRY(run(scd::Op::kPatchKV, jp.build(), model->dtype, stream));
      continue;
    }
    for (const auto& p : jp.build()) {
      const hipError_t e = scd::launch_patch_bf16(p, stream);
      if (e != hipSuccess) return fail(SCD_ERR_HIP, "patch launch failed: %s", hipGetErrorString(e));
    }
  }
  return ok();
}

}  // extern "C"

// ---- Offline Reuse fit ------------------------------------------------------------------------
namespace {

// Slices of the row axis for a Gram launch of n_jobs jobs: about two rounds of workgroups (the
// whole-Gram kernel fits one workgroup per CU, the tile kernels two) when the tiles allow, at
// least 512 rows per slice, slice lengths a multiple of the kernels' k-step.
int64_t fit_slices(int n_jobs, int w, bool bf16, int64_t n_rows, int64_t* slice_rows) {
  const int64_t units = scd::fit_units_per_slice(bf16, w, n_jobs);
  int64_t ns = (scd::fit_full_gram(bf16, w) ? 512 : 1024) / units;
  const int64_t max_ns = (n_rows + 511) / 512;
  if (ns > max_ns) ns = max_ns;
  if (ns < 1) ns = 1;
  int64_t sr = (n_rows + ns - 1) / ns;
  sr = (sr + scd::kFitRowStep - 1) / scd::kFitRowStep * scd::kFitRowStep;
  ns = (n_rows + sr - 1) / sr;
  if (ns < 1) ns = 1;
  *slice_rows = sr;
  return ns;
}

int count_reuse(const scd_model_t* m) {
  int n = 0;
  for (int l = 0; l < m->n_layers; ++l) n += m->is_patch[l] ? 0 : 1;
  return n;
}

size_t fit_gram_ws(const scd_model_t* m, int64_t n_rows) {
  const int R = count_reuse(m);
  size_t best = 0;
  for (int done = 0; done < R; done += scd::kMaxJobs) {
    const int jobs = R - done < scd::kMaxJobs ? R - done : scd::kMaxJobs;
    int64_t sr;
    const int64_t ns = fit_slices(jobs, m->basis_width, m->dtype == SCD_BF16, n_rows, &sr);
    const size_t b = static_cast<size_t>(jobs) * ns * scd::fit_upper_tiles(m->basis_width) *
                     (scd::kFitTile * scd::kFitTile + scd::kFitTile) * sizeof(float);
    if (b > best) best = b;
  }
  return best;
}

size_t fit_solve_ws(const scd_model_t* m) {
  const int R = count_reuse(m);
  const size_t jobs = R < scd::kMaxJobs ? R : scd::kMaxJobs;
  return jobs * static_cast<size_t>(scd::fit_solve_layer_doubles(m->basis_width)) * sizeof(double);
}

// Per-layer output buffers of the fit must be distinct: the layers of a launch are written
// concurrently.
scd_status_t distinct_outputs(const std::vector<int>& layers, const void* const* arr,
                              const char* name) {
  for (size_t i = 0; i < layers.size(); ++i)
    for (size_t j = 0; j < i; ++j)
      if (arr[layers[i]] == arr[layers[j]])
        return fail(SCD_ERR_SHAPE, "%s[%d] repeats layer %d's buffer", name, layers[i], layers[j]);
  return SCD_OK;
}

scd_status_t check_fit_model(const scd_model_t* model, int32_t branch) {
  SCD_TRY(check_model(model));
  if (branch != 0 && branch != 1)
    return fail(SCD_ERR_SHAPE, "branch must be 0 (keys) or 1 (values), got %d", branch);
  if (model->basis_width % 64 != 0)
    return fail(SCD_ERR_UNSUPPORTED, "the fit needs basis_width %% 64 == 0 (got %d)",
                model->basis_width);
  return SCD_OK;
}

}  // namespace

extern "C" {

size_t scd_fit_workspace_bytes(const scd_model_t* model, int64_t n_tokens) {
  if (check_model(model) != SCD_OK || n_tokens < 1) return 0;
  const int64_t g = kv_width(model) / model->basis_width;
  const size_t a = fit_gram_ws(model, n_tokens * g), b = fit_solve_ws(model);
  return a > b ? a : b;
}

scd_status_t scd_fit_gram(const scd_model_t* model, const scd_batch_t* batch,
                          const void* rope_table, int64_t max_position, int32_t branch,
                          const void* const* a_in, const void* const* b_in,
                          float* const* gram, float* const* colsum, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  SCD_TRY(check_fit_model(model, branch));
  SCD_TRY(check_batch(batch));
  if (batch->n_tokens < 1) return fail(SCD_ERR_SHAPE, "the fit needs at least one token");
  const int w = model->basis_width;
  const int g = static_cast<int>(kv_width(model) / w);
  const int64_t n_rows = batch->n_tokens * g;
  std::vector<int> layers;
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) continue;
    layers.push_back(l);
    SCD_TRY(need_ptr(a_in, l, "a_in"));
    SCD_TRY(need_ptr(b_in, l, "b_in"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(gram), l, "gram"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(colsum), l, "colsum"));
  }
  if (layers.empty()) return ok();
  SCD_TRY(distinct_outputs(layers, reinterpret_cast<const void* const*>(gram), "gram"));
  SCD_TRY(distinct_outputs(layers, reinterpret_cast<const void* const*>(colsum), "colsum"));
  if (branch == 0) SCD_TRY(check_rope(rope_table, max_position));
  if (workspace == nullptr) return fail(SCD_ERR_NULL, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SCD_ERR_ALIGN, "workspace is not 16-byte aligned");
  const size_t need = fit_gram_ws(model, n_rows);
  if (workspace_bytes < need)
    return fail(SCD_ERR_SHAPE, "workspace_bytes %zu < %zu needed", workspace_bytes, need);

  for (size_t done = 0; done < layers.size(); done += scd::kMaxJobs) {
    scd::FitGramParams p{};
    p.n_jobs = 0;
    for (size_t i = done; i < layers.size() && i < done + scd::kMaxJobs; ++i) {
      const int l = layers[i];
      p.jobs[p.n_jobs++] = {a_in[l], b_in[l], gram[l], colsum[l]};
    }
    p.w = w;
    p.n_rows = n_rows;
    p.g = g;
    p.head_dim = model->head_dim;
    p.derope = branch == 0 ? 1 : 0;
    p.n_slices = static_cast<int32_t>(
        fit_slices(p.n_jobs, w, model->dtype == SCD_BF16, n_rows, &p.slice_rows));
    p.n_seqs = batch->n_seqs;
    p.cu_seqlens = batch->cu_seqlens;
    p.pos0 = batch->pos0;
    p.rope = static_cast<const float2*>(rope_table);
    p.max_pos = max_position;
    p.partial = static_cast<float*>(workspace);
    const hipError_t e = scd::launch_fit_gram(model->dtype == SCD_BF16, p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "fit Gram launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

}  // extern "C"

namespace {

// Validates a fit-solve call (everything but the workspace) and lists the Reuse layers it fits.
scd_status_t check_fit_solve(const scd_model_t* model, int32_t branch, int64_t n_rows,
                             double ridge_lambda, int32_t center, const float* const* gram,
                             const float* const* colsum, void* const* w_enc, void* const* w_dec,
                             void* const* mu_enc, void* const* mu_dec, std::vector<int>* layers) {
  SCD_TRY(check_fit_model(model, branch));
  const int w = model->basis_width;
  if (w > scd::kFitMaxSolveWidth)
    return fail(SCD_ERR_UNSUPPORTED, "the fit's solve takes basis_width <= %d (got %d)",
                scd::kFitMaxSolveWidth, w);
  if (n_rows < 1) return fail(SCD_ERR_SHAPE, "n_rows must be >= 1");
  if (!(ridge_lambda >= 0.0) || ridge_lambda > 1e300)
    return fail(SCD_ERR_SHAPE, "ridge_lambda must be finite and >= 0");
  if (center != 0 && center != 1) return fail(SCD_ERR_SHAPE, "center must be 0 or 1");
  const int32_t* ranks = branch == 0 ? model->rank_k : model->rank_v;
  layers->clear();
  for (int l = 0; l < model->n_layers; ++l) {
    if (model->is_patch[l]) continue;
    layers->push_back(l);
    SCD_TRY(check_rank(branch == 0 ? "rank_k" : "rank_v", l, ranks[l], w));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(gram), l, "gram"));
    SCD_TRY(need_ptr(reinterpret_cast<const void* const*>(colsum), l, "colsum"));
    SCD_TRY(need_ptr(w_enc, l, "w_enc"));
    SCD_TRY(need_ptr(w_dec, l, "w_dec"));
    if (center) {
      SCD_TRY(need_ptr(mu_enc, l, "mu_enc"));
      SCD_TRY(need_ptr(mu_dec, l, "mu_dec"));
    }
  }
  if (layers->empty()) return SCD_OK;
  SCD_TRY(distinct_outputs(*layers, w_enc, "w_enc"));
  SCD_TRY(distinct_outputs(*layers, w_dec, "w_dec"));
  if (center) {
    SCD_TRY(distinct_outputs(*layers, mu_enc, "mu_enc"));
    SCD_TRY(distinct_outputs(*layers, mu_dec, "mu_dec"));
  }
  return SCD_OK;
}

// Launches the solve for `layers`, at most jobs_per_launch layers per launch, every launch using
// the same `work` matrices (launches on one stream run in order, so they never overlap).
scd_status_t enqueue_fit_solve(const scd_model_t* model, int32_t branch, int64_t n_rows,
                               double ridge_lambda, int32_t center, const float* const* gram,
                               const float* const* colsum, void* const* w_enc,
                               void* const* w_dec, void* const* mu_enc, void* const* mu_dec,
                               const std::vector<int>& layers, size_t jobs_per_launch,
                               double* work, hipStream_t stream) {
  const int32_t* ranks = branch == 0 ? model->rank_k : model->rank_v;
  for (size_t done = 0; done < layers.size(); done += jobs_per_launch) {
    scd::FitSolveParams p{};
    p.n_jobs = 0;
    for (size_t i = done; i < layers.size() && i < done + jobs_per_launch; ++i) {
      const int l = layers[i];
      p.jobs[p.n_jobs++] = {gram[l], colsum[l], w_enc[l], w_dec[l],
                            center ? mu_enc[l] : nullptr, center ? mu_dec[l] : nullptr, ranks[l], 0};
    }
    p.w = model->basis_width;
    p.n_rows = n_rows;
    p.lambda = ridge_lambda;
    p.center = center;
    p.bf16 = model->dtype == SCD_BF16 ? 1 : 0;
    p.work = work;
    const hipError_t e = scd::launch_fit_solve(p, stream);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "fit solve launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

}  // namespace

extern "C" {

scd_status_t scd_fit_solve(const scd_model_t* model, int32_t branch, int64_t n_rows,
                           double ridge_lambda, int32_t center, const float* const* gram,
                           const float* const* colsum, void* const* w_enc, void* const* w_dec,
                           void* const* mu_enc, void* const* mu_dec, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  std::vector<int> layers;
  SCD_TRY(check_fit_solve(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc, w_dec,
                          mu_enc, mu_dec, &layers));
  if (layers.empty()) return ok();
  if (workspace == nullptr) return fail(SCD_ERR_NULL, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SCD_ERR_ALIGN, "workspace is not 16-byte aligned");
  const size_t need = fit_solve_ws(model);
  if (workspace_bytes < need)
    return fail(SCD_ERR_SHAPE, "workspace_bytes %zu < %zu needed", workspace_bytes, need);
  return enqueue_fit_solve(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc,
                           w_dec, mu_enc, mu_dec, layers, scd::kMaxJobs,
                           static_cast<double*>(workspace), stream);
}

size_t scd_fit_solve_noalloc_max_bytes(void) { return scd::kFitScratchBytes; }

scd_status_t scd_fit_solve_noalloc(const scd_model_t* model, int32_t branch, int64_t n_rows,
                                   double ridge_lambda, int32_t center, const float* const* gram,
                                   const float* const* colsum, void* const* w_enc,
                                   void* const* w_dec, void* const* mu_enc, void* const* mu_dec,
                                   hipStream_t stream) {
  std::vector<int> layers;
  SCD_TRY(check_fit_solve(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc, w_dec,
                          mu_enc, mu_dec, &layers));
  if (layers.empty()) return ok();
  const size_t per_layer =
      static_cast<size_t>(scd::fit_solve_layer_doubles(model->basis_width)) * sizeof(double);
  if (per_layer > scd::kFitScratchBytes)
    return fail(SCD_ERR_WORKSPACE,
                "basis_width %d needs %zu bytes of solve scratch per layer; the allocation-free "
                "solve holds %zu",
                model->basis_width, per_layer, scd::kFitScratchBytes);
  double* work = nullptr;
  const hipError_t e = scd::fit_scratch(&work);
  if (e != hipSuccess)
    return fail(SCD_ERR_HIP, "scratch address lookup failed: %s", hipGetErrorString(e));
  size_t jobs = scd::kFitScratchBytes / per_layer;
  if (jobs > static_cast<size_t>(scd::kMaxJobs)) jobs = scd::kMaxJobs;
  return enqueue_fit_solve(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc,
                           w_dec, mu_enc, mu_dec, layers, jobs, work, stream);
}

}  // extern "C"
