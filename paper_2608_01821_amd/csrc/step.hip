// One denoising step (Sec. 3.1, Eq. 1) over a packed batch, and the workspace
// layout it uses.  The host side only validates, packs the per-sequence table
// and enqueues kernels; every arithmetic step runs on the GPU.
//
// Layer schedule (pre-norm, n_layers times):
//   A = RMSNorm(X)                 (fused into the assembly for layer 0, and
//                                   into the previous layer's tail otherwise)
//   QKV = A Wqkv^T                 GEMM, bf16 out
//   rotary embedding on Q, K       in place
//   O = attention(Q, K, V)         non-causal, per sequence
//   X += O Wo^T                    GEMM, fp32 residual epilogue
//   A = RMSNorm(X)
//   H = silu(A Wg^T) * (A Wu^T)    dual GEMM, SwiGLU epilogue
//   X += H Wd^T                    GEMM, fp32 residual epilogue
// then the final norm of the masked response rows, the vocabulary GEMM with
// the fused (max, argmax, sum-exp) reduction, and the merge across slabs.

#include <algorithm>
#include <vector>

#include "common.h"

namespace davet {

struct Layout {
  size_t flags;                        // 16-bit overflow counter (offset 0)
  size_t conf, argmax, argmax2;        // run_schedule scratch
  size_t X, A, QKV, O, H, rope, pos, list, slot, Hm, pmax, psum, parg, logits;
  size_t part;                         // split-K partial tiles (16-bit path)
  size_t rope_sched;                   // run_schedule's rotary table (last)
  size_t total;
};

// Bytes of fp32 partial tiles the 16-bit GEMMs of a step with at most
// `tokens` rows may need (the largest over the four projections).
static size_t partial_bytes(const davet_model_cfg& c, int64_t tokens) {
  if (!is16(c.dtype)) return 0;
  const int64_t Ns[4] = {3LL * c.d, c.d, 2LL * c.ffn, c.d};
  const int64_t Ks[4] = {c.d, c.d, c.d, c.ffn};
  size_t best = 0;
  for (int g = 0; g < 4; ++g)
    best = std::max(best, gemm16_partial_bound((int)tokens, (int)Ns[g], (int)Ks[g]));
  return best;
}

static Layout make_layout(const davet_model_cfg& c, int64_t tokens,
                          int64_t seqs, int64_t L) {
  const size_t es = dtype_size(c.dtype);
  const int64_t rows = seqs * L;
  const int64_t slabs = head16_slabs(c.vocab);
  Layout o{};
  size_t p = 0;
  auto take = [&](size_t bytes) {
    const size_t at = p;
    p = align_up(p + bytes, 256);
    return at;
  };
  o.flags = take(256);
  o.conf = take(rows * 4);
  o.argmax = take(rows * 4);
  o.argmax2 = take(rows * 4);    // the schedule loop's previous predictions
  o.X = take((size_t)tokens * c.d * 4);
  o.A = take((size_t)tokens * c.d * es);
  o.QKV = take((size_t)tokens * 3 * c.d * es);
  o.O = take((size_t)tokens * c.d * es);
  o.H = take((size_t)tokens * c.ffn * es);
  o.rope = take((size_t)tokens * (c.head_dim / 2) * 8);
  o.pos = take((size_t)tokens * 4);
  o.list = take((size_t)(rows + 1) * 4);
  o.slot = take((size_t)rows * 4);
  o.Hm = take((size_t)rows * c.d * es);
  if (is16(c.dtype)) {
    o.pmax = take((size_t)rows * slabs * 4);
    o.psum = take((size_t)rows * slabs * 4);
    o.parg = take((size_t)rows * slabs * 4);
    o.logits = 0;
  } else {
    o.logits = take((size_t)rows * c.vocab * 4);
  }
  // split-K partials of the projections, and (not live at the same time)
  // the key-range partials of attention
  o.part = take(is16(c.dtype)
                    ? std::max(partial_bytes(c, tokens),
                               attention_part_bytes(tokens, seqs, c.n_heads))
                    : 0);
  // Every region above grows with the token count, so a step with fewer
  // tokens than the workspace was sized for never reaches this one: the
  // schedule loop keeps its rotary table here for all its steps.
  o.rope_sched = take((size_t)tokens * (c.head_dim / 2) * 8);
  o.total = p;
  return o;
}

// null counts as aligned (optional vectors)
static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

static int check_cfg(const davet_model_cfg* c) {
  DAVET_CHECK_ARG(c, DAVET_EINVAL, "model cfg is null");
  DAVET_CHECK_ARG(c->dtype == DAVET_F32 || is16(c->dtype), DAVET_EDTYPE,
                  "cfg.dtype must be DAVET_F32, DAVET_BF16 or DAVET_F16");
  DAVET_CHECK_ARG(c->n_layers >= 0 && c->n_heads >= 1, DAVET_ESHAPE,
                  "cfg: n_layers >= 0 and n_heads >= 1 required");
  DAVET_CHECK_ARG(c->head_dim == 64 || c->head_dim == 128, DAVET_ESHAPE,
                  "cfg.head_dim must be 64 or 128");
  DAVET_CHECK_ARG(c->d == c->n_heads * c->head_dim, DAVET_ESHAPE,
                  "cfg.d must equal n_heads * head_dim");
  DAVET_CHECK_ARG(c->d <= 8192 && c->ffn >= 1, DAVET_ESHAPE,
                  "cfg.d must be <= 8192, ffn >= 1");
  DAVET_CHECK_ARG(c->vocab >= 2 && c->mask_id >= 0 && c->mask_id < c->vocab,
                  DAVET_ESHAPE, "cfg: vocab >= 2 and 0 <= mask_id < vocab");
  DAVET_CHECK_ARG(c->rms_eps >= 0.f && c->rope_theta > 0.f, DAVET_EINVAL,
                  "cfg: rms_eps >= 0 and rope_theta > 0 required");
  if (is16(c->dtype)) {
    DAVET_CHECK_ARG(c->head_dim == 128, DAVET_ESHAPE,
                    "16-bit path: head_dim must be 128");
    DAVET_CHECK_ARG(c->d % 128 == 0 && c->ffn % 64 == 0 && (3 * c->d) % 128 == 0,
                    DAVET_ESHAPE, "16-bit path: d % 128 == 0 and ffn % 64 == 0");
  }
  return DAVET_OK;
}

int workspace_layout_bytes(const davet_model_cfg* c, int64_t tokens,
                           int64_t seqs, int64_t L, size_t* out) {
  *out = make_layout(*c, tokens, seqs, L).total;
  return DAVET_OK;
}

// Used by run_schedule to reach its scratch region.
void schedule_scratch(const davet_model_cfg* c, int64_t tokens, int64_t seqs,
                      int64_t L, size_t* conf_off, size_t* argmax_off,
                      size_t* argmax2_off, size_t* rope_off) {
  const Layout o = make_layout(*c, tokens, seqs, L);
  *conf_off = o.conf;
  *argmax_off = o.argmax;
  *argmax2_off = o.argmax2;
  *rope_off = o.rope_sched;
}

}  // namespace davet

extern "C" int davet_workspace_bytes(const davet_model_cfg* cfg,
                                     int32_t max_tokens, int32_t max_seqs,
                                     int32_t L, size_t* bytes) {
  using namespace davet;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  DAVET_CHECK_ARG(bytes, DAVET_EINVAL, "davet_workspace_bytes: bytes is null");
  DAVET_CHECK_ARG(max_tokens >= 1 && max_seqs >= 1 &&
                      max_seqs <= DAVET_MAX_SEQS && L >= 1 && L <= DAVET_MAX_RESP,
                  DAVET_ESHAPE, "davet_workspace_bytes: sizes out of range");
  return workspace_layout_bytes(cfg, max_tokens, max_seqs, L, bytes);
}

namespace davet {
int denoise_step_impl(const davet_model_cfg* cfg, const davet_weights* w,
                      int32_t n_seqs, const void* const* view_ptrs,
                      const int32_t* n_view, const int32_t* prompt_ids,
                      const int32_t* cu_prompt, const int32_t* resp_ids,
                      const uint8_t* resp_masked, int32_t L, float* conf_out,
                      int32_t* argmax_out, float* logits_out, void* workspace,
                      size_t ws_bytes, const float* rope_cs, int rows_bound,
                      int clear_overflow, hipStream_t stream);
}  // namespace davet

extern "C" int davet_denoise_step(const davet_model_cfg* cfg,
                                  const davet_weights* w, int32_t n_seqs,
                                  const void* const* view_ptrs,
                                  const int32_t* n_view,
                                  const int32_t* prompt_ids,
                                  const int32_t* cu_prompt,
                                  const int32_t* resp_ids,
                                  const uint8_t* resp_masked, int32_t L,
                                  float* conf_out, int32_t* argmax_out,
                                  float* logits_out, void* workspace,
                                  size_t ws_bytes, hipStream_t stream) {
  return davet::denoise_step_impl(cfg, w, n_seqs, view_ptrs, n_view,
                                  prompt_ids, cu_prompt, resp_ids, resp_masked,
                                  L, conf_out, argmax_out, logits_out,
                                  workspace, ws_bytes, nullptr, n_seqs * L,
                                  1, stream);
}

extern "C" int davet_fp16_overflow_count(const void* workspace, int32_t* count,
                                         hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(workspace && count, DAVET_EINVAL,
                  "davet_fp16_overflow_count: null pointer");
  DAVET_CHECK_ARG(((uintptr_t)workspace & 255) == 0, DAVET_EINVAL,
                  "davet_fp16_overflow_count: workspace must be 256-byte aligned");
  // the counter sits at offset 0 of every workspace layout
  DAVET_HIP(hipMemcpyAsync(count, workspace, sizeof(int32_t),
                         hipMemcpyDeviceToHost, stream));
  DAVET_HIP(hipStreamSynchronize(stream));
  return DAVET_OK;
}

// rope_cs: a rotary table already holding every position this step uses
// (the schedule loop's); null: build it in the step's own region.
// rows_bound: an upper bound on the masked positions the caller knows on the
// host (n_seqs * L when it knows none); it only sizes the head's grid, whose
// workgroups still loop over any live rows beyond it.
// clear_overflow: zero the workspace's overflow counter before this step's
// stores (a schedule keeps counting over all its steps).
int davet::denoise_step_impl(const davet_model_cfg* cfg, const davet_weights* w,
                             int32_t n_seqs, const void* const* view_ptrs,
                             const int32_t* n_view, const int32_t* prompt_ids,
                             const int32_t* cu_prompt, const int32_t* resp_ids,
                             const uint8_t* resp_masked, int32_t L,
                             float* conf_out, int32_t* argmax_out,
                             float* logits_out, void* workspace,
                             size_t ws_bytes, const float* rope_cs,
                             int rows_bound, int clear_overflow,
                             hipStream_t stream) {
  using namespace davet;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  const davet_model_cfg& c = *cfg;
  DAVET_CHECK_ARG(w && w->embed && w->head, DAVET_EINVAL,
                  "davet_denoise_step: null weights");
  DAVET_CHECK_ARG(c.n_layers == 0 || w->layers, DAVET_EINVAL,
                  "davet_denoise_step: null layer table");
  for (int l = 0; l < c.n_layers; ++l) {
    const davet_layer_weights& lw = w->layers[l];
    DAVET_CHECK_ARG(lw.wqkv && lw.wo && lw.wg && lw.wu && lw.wd, DAVET_EINVAL,
                    "davet_denoise_step: null layer weight");
    DAVET_CHECK_ARG(aligned16(lw.wqkv) && aligned16(lw.wo) && aligned16(lw.wg) &&
                        aligned16(lw.wu) && aligned16(lw.wd) &&
                        aligned16(lw.attn_norm) && aligned16(lw.ffn_norm),
                    DAVET_EINVAL,
                    "davet_denoise_step: layer weights must be 16-byte aligned");
  }
  DAVET_CHECK_ARG(aligned16(w->embed) && aligned16(w->head) &&
                      aligned16(w->final_norm),
                  DAVET_EINVAL,
                  "davet_denoise_step: weights must be 16-byte aligned");
  DAVET_CHECK_ARG(w->head_layout == DAVET_HEAD_ROWS ||
                      (w->head_layout == DAVET_HEAD_TILED && is16(c.dtype)),
                  DAVET_EINVAL,
                  "davet_denoise_step: head_layout must be DAVET_HEAD_ROWS, or "
                  "DAVET_HEAD_TILED with a 16-bit model");
  DAVET_CHECK_ARG(n_seqs >= 1 && n_seqs <= DAVET_MAX_SEQS, DAVET_ESHAPE,
                  "davet_denoise_step: n_seqs out of range [1, 64]");
  DAVET_CHECK_ARG(L >= 1 && L <= DAVET_MAX_RESP, DAVET_ESHAPE,
                  "davet_denoise_step: L out of range [1, 1024]");
  DAVET_CHECK_ARG(view_ptrs && n_view && cu_prompt && resp_ids && resp_masked &&
                      conf_out && argmax_out && workspace,
                  DAVET_EINVAL, "davet_denoise_step: null pointer");
  DAVET_CHECK_ARG(cu_prompt[0] == 0, DAVET_ESHAPE,
                  "davet_denoise_step: cu_prompt[0] must be 0");
  DAVET_CHECK_ARG(((uintptr_t)workspace & 255) == 0, DAVET_ENOMEM,
                  "davet_denoise_step: workspace must be 256-byte aligned");

  SeqPack sp{};
  ViewPtrs vp{};
  sp.n_seqs = n_seqs;
  sp.L = L;
  int64_t total = 0;
  int max_n = 0;
  for (int s = 0; s < n_seqs; ++s) {
    DAVET_CHECK_ARG(n_view[s] >= 0, DAVET_ESHAPE,
                    "davet_denoise_step: negative view length");
    DAVET_CHECK_ARG(n_view[s] == 0 || view_ptrs[s], DAVET_EINVAL,
                    "davet_denoise_step: null view pointer");
    DAVET_CHECK_ARG(aligned16(view_ptrs[s]), DAVET_EINVAL,
                    "davet_denoise_step: view pointers must be 16-byte aligned");
    const int plen = cu_prompt[s + 1] - cu_prompt[s];
    DAVET_CHECK_ARG(plen >= 0, DAVET_ESHAPE,
                    "davet_denoise_step: cu_prompt must be non-decreasing");
    DAVET_CHECK_ARG(plen == 0 || prompt_ids, DAVET_EINVAL,
                    "davet_denoise_step: null prompt_ids");
    const int64_t n = (int64_t)n_view[s] + plen + L;
    sp.row0[s] = (int32_t)total;
    sp.nview[s] = n_view[s];
    sp.pstart[s] = cu_prompt[s];
    sp.plen[s] = plen;
    vp.p[s] = view_ptrs[s];
    total += n;
    max_n = std::max<int64_t>(max_n, n);
    DAVET_CHECK_ARG(total < (1ll << 30), DAVET_ESHAPE,
                    "davet_denoise_step: too many tokens");
  }
  sp.row0[n_seqs] = (int32_t)total;
  sp.total = (int32_t)total;
  const Layout lay = make_layout(c, total, n_seqs, L);
  DAVET_CHECK_ARG(ws_bytes >= lay.total, DAVET_ENOMEM,
                  "davet_denoise_step: workspace too small (" +
                      std::to_string(ws_bytes) + " < " +
                      std::to_string(lay.total) + " bytes)");

  char* ws = static_cast<char*>(workspace);
  float* X = reinterpret_cast<float*>(ws + lay.X);
  void* A = ws + lay.A;
  void* QKV = ws + lay.QKV;
  void* O = ws + lay.O;
  void* H = ws + lay.H;
  const float* rope = rope_cs ? rope_cs : reinterpret_cast<float*>(ws + lay.rope);
  int32_t* pos = reinterpret_cast<int32_t*>(ws + lay.pos);
  float* part = reinterpret_cast<float*>(ws + lay.part);
  const size_t part_cap = partial_bytes(c, total);
  // the partial region ends where the schedule's rotary table begins
  const size_t attn_part_cap = lay.rope_sched - lay.part;
  int32_t* list = reinterpret_cast<int32_t*>(ws + lay.list);
  int32_t* slot = reinterpret_cast<int32_t*>(ws + lay.slot);
  void* Hm = ws + lay.Hm;
  const int rows = n_seqs * L;
  const bool bf = is16(c.dtype);
  const int dt = c.dtype;
  const int d = c.d, F = c.ffn;
  hipStream_t s = stream;

#define RUN(x) do { int rc_ = (x); if (rc_) return rc_; } while (0)
  if (!rope_cs)
    RUN(launch_rope_table(max_n, c.head_dim, c.rope_theta,
                          reinterpret_cast<float*>(ws + lay.rope), s));
  const float* g0 = c.n_layers > 0 ? w->layers[0].attn_norm : w->final_norm;
  int32_t* overflow = reinterpret_cast<int32_t*>(ws + lay.flags);
  const RowList rl{n_seqs * L, list,     conf_out,      argmax_out,
                   slot,       overflow, clear_overflow};
  RUN(launch_assemble_norm(sp, vp, c.dtype, w->embed, prompt_ids, resp_ids,
                           resp_masked, c.mask_id, c.vocab, d, g0, c.rms_eps, X, A,
                           pos, rl, s));
  const int T = sp.total;
  const GemmPlan p_qkv = plan_gemm16(T, 3 * d, d), p_o = plan_gemm16(T, d, d);
  const GemmPlan p_gu = plan_gemm16(T, 2 * F, d), p_dn = plan_gemm16(T, d, F);
  bool a_ready = true;       // A holds RMSNorm(X) for the next GEMM
  bool hm_ready = false;     // Hm holds the final norm of the masked rows
  for (int l = 0; l < c.n_layers; ++l) {
    const davet_layer_weights& lw = w->layers[l];
    if (!a_ready) RUN(launch_rmsnorm(X, T, d, lw.attn_norm, c.rms_eps,
                                     c.dtype, A, s));
    if (bf) {
      const uint16_t* Ah = (const uint16_t*)A;
      // QKV projection, rotary embedding on the query and key columns
      RUN(launch_gemm16(dt, EPI_STORE, p_qkv, Ah, (const uint16_t*)lw.wqkv,
                        nullptr, QKV, T, 3 * d, d, 3 * d, pos, rope, 2 * d,
                        part, part_cap, KC_GEMM_QKV, s, overflow));
      if (p_qkv.ksplit > 1)
        RUN(launch_reduce_store_rope(dt, part, p_qkv.ksplit, T, 3 * d, 2 * d,
                                     pos, rope, QKV, s, overflow));
      RUN(launch_attention16(dt, (const uint16_t*)QKV, (uint16_t*)O, sp,
                             c.n_heads, c.head_dim, part, attn_part_cap, s));
      // X += O Wo^T, then A = RMSNorm(X) for the feed-forward block
      RUN(launch_gemm16(dt, EPI_ADD_F32, p_o, (const uint16_t*)O,
                        (const uint16_t*)lw.wo, nullptr, X, T, d, d, d,
                        nullptr, nullptr, 0, part, part_cap, KC_GEMM_O, s));
      if (p_o.ksplit > 1)
        RUN(launch_reduce_add_norm(dt, part, p_o.ksplit, T, d, X, lw.ffn_norm,
                                   c.rms_eps, A, s));
      else
        RUN(launch_rmsnorm(X, T, d, lw.ffn_norm, c.rms_eps, c.dtype, A, s));
      RUN(launch_gemm16(dt, EPI_SWIGLU, p_gu, Ah, (const uint16_t*)lw.wg,
                        (const uint16_t*)lw.wu, H, T, 2 * F, d, F, nullptr,
                        nullptr, 0, part, part_cap, KC_GEMM_GATEUP, s,
                        overflow));
      if (p_gu.ksplit > 1)
        RUN(launch_reduce_swiglu(dt, part, p_gu.ksplit, T, F, H, s, overflow));
      // X += H Wd^T (and the next layer's input norm when reducing splits)
      RUN(launch_gemm16(dt, EPI_ADD_F32, p_dn, (const uint16_t*)H,
                        (const uint16_t*)lw.wd, nullptr, X, T, d, F, d,
                        nullptr, nullptr, 0, part, part_cap, KC_GEMM_DOWN, s));
      a_ready = false;
      if (p_dn.ksplit > 1) {
        // and the next layer's input norm, or after the last layer the final
        // norm of the masked rows gathered into Hm
        if (l + 1 < c.n_layers) {
          RUN(launch_reduce_add_norm(dt, part, p_dn.ksplit, T, d, X,
                                     w->layers[l + 1].attn_norm, c.rms_eps, A,
                                     s));
          a_ready = true;
        } else {
          RUN(launch_reduce_add_gather(dt, part, p_dn.ksplit, T, d, X, sp,
                                       slot, w->final_norm, c.rms_eps, Hm, s));
          hm_ready = true;
        }
      }
    } else {
      RUN(launch_gemm_f32(EPI_STORE, (const float*)A, (const float*)lw.wqkv,
                          nullptr, (float*)QKV, sp.total, 3 * d, d, 3 * d,
                          KC_GEMM_F32, nullptr, s));
      RUN(launch_rope(QKV, sp.total, c.n_heads, c.head_dim, c.dtype, sp, rope, s));
      RUN(launch_attention_f32((const float*)QKV, (float*)O, sp, c.n_heads,
                               c.head_dim, s));
      RUN(launch_gemm_f32(EPI_ADD_F32, (const float*)O, (const float*)lw.wo,
                          nullptr, X, sp.total, d, d, d, KC_GEMM_F32, nullptr, s));
      RUN(launch_rmsnorm(X, sp.total, d, lw.ffn_norm, c.rms_eps, c.dtype, A, s));
      RUN(launch_gemm_f32(EPI_SWIGLU, (const float*)A, (const float*)lw.wg,
                          (const float*)lw.wu, (float*)H, sp.total, F, d, F,
                          KC_GEMM_F32, nullptr, s));
      RUN(launch_gemm_f32(EPI_ADD_F32, (const float*)H, (const float*)lw.wd,
                          nullptr, X, sp.total, d, F, d, KC_GEMM_F32, nullptr, s));
      a_ready = false;
    }
  }
  if (!hm_ready)
    RUN(launch_final_norm_gather(X, sp, list, rows, d, w->final_norm,
                                 c.rms_eps, c.dtype, Hm, s));
  if (bf) {
    const bool tiled = w->head_layout == DAVET_HEAD_TILED;
    const int live = std::max(1, std::min(rows, rows_bound));
    const int slabs = head16_slabs(c.vocab, tiled, live);
    float* pmax = reinterpret_cast<float*>(ws + lay.pmax);
    float* psum = reinterpret_cast<float*>(ws + lay.psum);
    int32_t* parg = reinterpret_cast<int32_t*>(ws + lay.parg);
    RUN(launch_head16(dt, (const uint16_t*)Hm, (const uint16_t*)w->head, list,
                      rows, c.vocab, d, c.mask_id, pmax, psum, parg,
                      logits_out, s, tiled, live));
    RUN(launch_head_merge(list, rows, slabs, pmax, psum, parg, conf_out,
                          argmax_out, s));
  } else {
    float* logits = reinterpret_cast<float*>(ws + lay.logits);
    RUN(launch_gemm_f32(EPI_STORE, (const float*)Hm, (const float*)w->head,
                        nullptr, logits, rows, c.vocab, d, c.vocab, KC_HEAD,
                        list, s));
    RUN(launch_head_reduce_f32(logits, list, rows, c.vocab, c.mask_id,
                               conf_out, argmax_out, logits_out, s));
  }
#undef RUN
  return DAVET_OK;
}
