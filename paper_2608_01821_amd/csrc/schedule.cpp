// The DAVET loop (Sec. 3.1 with Sec. 4; the procedure of Fig. 2): views are
// built once per sample, then every step picks each sample's level (a fixed
// schedule, or the allocation policy from the previous step's signals), runs
// the denoiser and commits.  In policy mode the GPU forms the risk signals
// and the next allocation after each commitment (launch_policy_step) and
// writes the next levels and budgets into the caller's mailbox (pinned,
// host-coherent memory from davet_mailbox_create), then a stamp; the host
// polls the stamp (the only crossing per step: the next step's launch sizes
// depend on the levels) and enqueues the next step.  The loop itself
// allocates and frees nothing.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstddef>
#include <string>
#include <vector>

#include "common.h"

// What the device policy step publishes for the host (one per mailbox).
struct davet_mailbox {
  struct Data {
    int32_t level[DAVET_MAX_SEQS];
    double budget[DAVET_MAX_SEQS];
    int32_t done;                    // stamp of the last step published
  };
  Data* host = nullptr;              // pinned, host-coherent
  Data* dev = nullptr;               // its device address
  uint32_t next_stamp = 1;           // stamps are unique per mailbox
};

namespace davet {
void schedule_scratch(const davet_model_cfg* c, int64_t tokens, int64_t seqs,
                      int64_t L, size_t* conf_off, size_t* argmax_off,
                      size_t* argmax2_off, size_t* rope_off);
int launch_policy_step(int n_seqs, int L, int K, const double* alpha,
                       const double* lower, const double* upper,
                       const float* conf, const int32_t* argmax,
                       const int32_t* argmax_prev, const uint8_t* masked_after,
                       int32_t* level_out, double* budget_out, double* r_out,
                       double* cbar_out, double* churn_out, int32_t* done,
                       int32_t stamp, hipStream_t s);
int denoise_step_impl(const davet_model_cfg* cfg, const davet_weights* w,
                      int32_t n_seqs, const void* const* view_ptrs,
                      const int32_t* n_view, const int32_t* prompt_ids,
                      const int32_t* cu_prompt, const int32_t* resp_ids,
                      const uint8_t* resp_masked, int32_t L, float* conf_out,
                      int32_t* argmax_out, float* logits_out, void* workspace,
                      size_t ws_bytes, const float* rope_cs, int rows_bound,
                      int clear_overflow, hipStream_t stream);

// Host-side limit on one wait for a step's published levels (seconds).
static std::atomic<double> g_wait_limit_s{120.0};

// Waits until the GPU has published `want` to the pinned word *flag.  Polls
// the word (its writer fences at system scope first, so the data it guards
// is complete) and, every few thousand polls, the stream and the clock: an
// error on the stream, a stream that drained without the stamp, or a wait
// longer than the limit ends it with DAVET_EHIP.  After a time-out the
// step's kernels may still be running and will still write the mailbox.
static int wait_stamp(const volatile int32_t* flag, int32_t want,
                      hipStream_t s) {
  using clock = std::chrono::steady_clock;
  const auto t0 = clock::now();
  const double limit = g_wait_limit_s.load(std::memory_order_relaxed);
  for (unsigned spin = 1;; ++spin) {
    if (*flag == want) break;
    __builtin_ia32_pause();
    if ((spin & 4095) == 0) {
      const hipError_t q = hipStreamQuery(s);
      if (q != hipSuccess && q != hipErrorNotReady)
        return set_error(DAVET_EHIP, std::string("davet_run_schedule: ") +
                                         hipGetErrorString(q));
      if (q == hipSuccess && *flag != want)
        return set_error(DAVET_EHIP, "davet_run_schedule: the policy step "
                                     "ended without publishing its levels");
      const double waited =
          std::chrono::duration<double>(clock::now() - t0).count();
      if (waited > limit && *flag != want)
        return set_error(
            DAVET_EHIP,
            "davet_run_schedule: no levels published within " +
                std::to_string(limit) +
                " s (the stream is still running; synchronise it before "
                "reusing or destroying the mailbox)");
    }
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return DAVET_OK;
}
}  // namespace davet

extern "C" int davet_mailbox_create(davet_mailbox** out) {
  using namespace davet;
  DAVET_CHECK_ARG(out, DAVET_EINVAL, "davet_mailbox_create: out is null");
  *out = nullptr;
  davet_mailbox* mb = new (std::nothrow) davet_mailbox();
  DAVET_CHECK_ARG(mb, DAVET_ENOMEM, "davet_mailbox_create: out of host memory");
  hipError_t e = hipHostMalloc((void**)&mb->host, sizeof(davet_mailbox::Data),
                               hipHostMallocCoherent);
  if (e == hipSuccess)
    e = hipHostGetDevicePointer((void**)&mb->dev, mb->host, 0);
  if (e != hipSuccess) {
    if (mb->host) (void)hipHostFree(mb->host);
    delete mb;
    return set_error(DAVET_EHIP, std::string("davet_mailbox_create: ") +
                                     hipGetErrorString(e));
  }
  mb->host->done = 0;
  *out = mb;
  return DAVET_OK;
}

extern "C" int davet_mailbox_destroy(davet_mailbox* mb) {
  using namespace davet;
  if (!mb) return DAVET_OK;
  // a policy step still queued on some stream may write the mailbox
  const hipError_t e1 = hipDeviceSynchronize();
  const hipError_t e2 = hipHostFree(mb->host);
  delete mb;
  if (e1 != hipSuccess || e2 != hipSuccess)
    return set_error(DAVET_EHIP, std::string("davet_mailbox_destroy: ") +
                                     hipGetErrorString(e1 != hipSuccess ? e1 : e2));
  return DAVET_OK;
}

extern "C" int davet_set_wait_limit(double seconds) {
  using namespace davet;
  DAVET_CHECK_ARG(seconds > 0.0 && std::isfinite(seconds), DAVET_EINVAL,
                  "davet_set_wait_limit: seconds must be positive and finite");
  g_wait_limit_s.store(seconds, std::memory_order_relaxed);
  return DAVET_OK;
}

extern "C" int davet_run_schedule(
    const davet_model_cfg* cfg, const davet_weights* w, int32_t n_seqs,
    const davet_view_geom* geoms, const void* const* visual,
    void* const* view_bufs, const int32_t* prompt_ids, const int32_t* cu_prompt,
    int32_t L, int32_t T, int32_t k, const davet_policy* pols,
    const int32_t* fixed_levels, int32_t* resp_ids, uint8_t* resp_masked,
    int32_t* levels_out, double* budgets_out, float* conf_trace,
    int32_t* argmax_trace, davet_mailbox* mailbox, void* workspace,
    size_t ws_bytes, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(cfg && w && geoms && visual && cu_prompt && resp_ids &&
                      resp_masked && workspace,
                  DAVET_EINVAL, "davet_run_schedule: null argument");
  DAVET_CHECK_ARG(n_seqs >= 1 && n_seqs <= DAVET_MAX_SEQS, DAVET_ESHAPE,
                  "davet_run_schedule: n_seqs out of range");
  DAVET_CHECK_ARG(T >= 1 && k >= 1, DAVET_EINVAL,
                  "davet_run_schedule: T >= 1 and k >= 1 required");
  DAVET_CHECK_ARG((pols == nullptr) != (fixed_levels == nullptr), DAVET_EINVAL,
                  "davet_run_schedule: give exactly one of pols, fixed_levels");
  DAVET_CHECK_ARG(L >= 1 && L <= DAVET_MAX_RESP, DAVET_ESHAPE,
                  "davet_run_schedule: L out of range");
  DAVET_CHECK_ARG(!pols || T == 1 || mailbox, DAVET_EINVAL,
                  "davet_run_schedule: policy mode needs a mailbox "
                  "(davet_mailbox_create)");
  const int K = geoms[0].K;
  DAVET_CHECK_ARG(K >= 1 && K <= DAVET_MAX_LEVELS, DAVET_ESHAPE,
                  "davet_run_schedule: K out of range");
  DAVET_CHECK_ARG(K == 1 || view_bufs, DAVET_EINVAL,
                  "davet_run_schedule: view_bufs is null");

  // views: level pointers and sizes per sequence
  std::vector<const void*> lvl_ptr((size_t)n_seqs * K);
  std::vector<int32_t> lvl_n((size_t)n_seqs * K);
  int64_t max_tokens = 0, max_len = 0;
  for (int s = 0; s < n_seqs; ++s) {
    const davet_view_geom& g = geoms[s];
    DAVET_CHECK_ARG(g.K == K && g.d == cfg->d && g.dtype == cfg->dtype,
                    DAVET_ESHAPE,
                    "davet_run_schedule: geometry K/d/dtype must match cfg");
    int rc = davet_view_sizes(&g, &lvl_n[(size_t)s * K]);
    if (rc) return rc;
    for (int l = 0; l < K; ++l)
      lvl_ptr[(size_t)s * K + l] =
          l == K - 1 ? visual[s] : view_bufs[(size_t)s * (K - 1) + l];
    const int64_t len =
        lvl_n[(size_t)s * K + K - 1] + (cu_prompt[s + 1] - cu_prompt[s]) + L;
    max_tokens += len;
    max_len = std::max(max_len, len);
  }
  if (fixed_levels)
    for (int i = 0; i < n_seqs * T; ++i)
      DAVET_CHECK_ARG(fixed_levels[i] >= 0 && fixed_levels[i] < K, DAVET_EINVAL,
                      "davet_run_schedule: fixed level out of range");
  size_t need = 0;
  {
    int rc = davet_workspace_bytes(cfg, (int32_t)max_tokens, n_seqs, L, &need);
    if (rc) return rc;
  }
  DAVET_CHECK_ARG(ws_bytes >= need, DAVET_ENOMEM,
                  "davet_run_schedule: workspace smaller than the full-view size");
  size_t conf_off = 0, am_off = 0, am2_off = 0, rope_off = 0;
  schedule_scratch(cfg, max_tokens, n_seqs, L, &conf_off, &am_off, &am2_off,
                   &rope_off);
  char* ws = static_cast<char*>(workspace);

  // a1: evidence views, once per sample (the prune / merge realizers use the
  // start of the workspace as scratch; nothing else lives there yet)
  for (int s = 0; s < n_seqs; ++s) {
    std::vector<void*> lv(K, nullptr);
    for (int l = 0; l < K - 1; ++l) lv[l] = view_bufs[(size_t)s * (K - 1) + l];
    int rc = davet_build_views(&geoms[s], visual[s], lv.data(), nullptr,
                               nullptr, workspace, ws_bytes, stream);
    if (rc) return rc;
  }

  // rotary table for every position of the longest sequence, once per loop
  // (a step's sequences are never longer than at the full view)
  float* rope = reinterpret_cast<float*>(ws + rope_off);
  {
    int rc = launch_rope_table((int)max_len, cfg->head_dim, cfg->rope_theta,
                               rope, stream);
    if (rc) return rc;
  }

  // policy state: envelopes on the host (once per sample), the per-step
  // signals and allocation on the GPU, the next levels in the mailbox
  std::vector<double> lower, upper, alpha(n_seqs), lo_t(n_seqs), up_t(n_seqs);
  uint32_t stamp0 = 0;
  if (pols) {
    lower.resize((size_t)n_seqs * T);
    upper.resize((size_t)n_seqs * T);
    for (int s = 0; s < n_seqs; ++s) {
      DAVET_CHECK_ARG(pols[s].K == K, DAVET_EINVAL,
                      "davet_run_schedule: policy K must match the views");
      int rc = davet_policy_envelope(&pols[s], T, &lower[(size_t)s * T],
                                     &upper[(size_t)s * T]);
      if (rc) return rc;
      alpha[s] = pols[s].alpha;
    }
    if (T > 1) {
      // this call's stamps: stamp0 + t for t = 1..T-1, never reused by the
      // mailbox, so a late write of an earlier (failed) call cannot pass
      stamp0 = mailbox->next_stamp;
      mailbox->next_stamp += (uint32_t)T;
      if (mailbox->next_stamp > 0x7fff0000u) mailbox->next_stamp = 1;
    }
  }
  int32_t* am_buf[2] = {reinterpret_cast<int32_t*>(ws + am_off),
                        reinterpret_cast<int32_t*>(ws + am2_off)};
  std::vector<const void*> vptr(n_seqs);
  std::vector<int32_t> nview(n_seqs);

  for (int t = 1; t <= T; ++t) {
    for (int s = 0; s < n_seqs; ++s) {
      int lv;
      double b = NAN;
      if (pols && t == 1) {
        // r_1 = 1: no signal exists yet (Eq. 7)
        int rc = davet_policy_step(&pols[s], 1, T, &lower[(size_t)s * T],
                                   &upper[(size_t)s * T], 0.0, 0.0, &b, &lv,
                                   nullptr);
        if (rc) return rc;
      } else if (pols) {
        lv = mailbox->host->level[s];
        b = mailbox->host->budget[s];
        DAVET_CHECK_ARG(lv >= 0 && lv < K, DAVET_EHIP,
                        "davet_run_schedule: device policy returned a level "
                        "out of range");
      } else {
        lv = fixed_levels[(size_t)s * T + (t - 1)];
      }
      if (levels_out) levels_out[(size_t)s * T + (t - 1)] = lv;
      if (budgets_out) budgets_out[(size_t)s * T + (t - 1)] = b;
      vptr[s] = lvl_ptr[(size_t)s * K + lv];
      nview[s] = lvl_n[(size_t)s * K + lv];
    }
    float* conf = conf_trace ? conf_trace + (size_t)(t - 1) * n_seqs * L
                             : reinterpret_cast<float*>(ws + conf_off);
    int32_t* am = argmax_trace ? argmax_trace + (size_t)(t - 1) * n_seqs * L
                               : am_buf[(t - 1) & 1];
    // every step commits min(k, masked) positions per sequence, so before
    // step t at most max(0, L - k(t-1)) of a sequence's positions are masked
    const int64_t per_seq = std::max<int64_t>(0, (int64_t)L - (int64_t)k * (t - 1));
    const int rows_bound = (int)std::max<int64_t>(1, per_seq * n_seqs);
    int rc = denoise_step_impl(cfg, w, n_seqs, vptr.data(), nview.data(),
                               prompt_ids, cu_prompt, resp_ids, resp_masked, L,
                               conf, am, nullptr, workspace, ws_bytes, rope,
                               rows_bound, t == 1, stream);
    if (rc) return rc;
    rc = davet_unmask(n_seqs, L, k, conf, am, resp_ids, resp_masked, nullptr,
                      stream);
    if (rc) return rc;
    if (pols && t < T) {
      // signals of step t -> allocation of step t+1 (Sec. 4.2)
      const int32_t* am_prev =
          t == 1 ? nullptr
                 : argmax_trace ? argmax_trace + (size_t)(t - 2) * n_seqs * L
                                : am_buf[t & 1];
      for (int s = 0; s < n_seqs; ++s) {
        lo_t[s] = lower[(size_t)s * T + t];
        up_t[s] = upper[(size_t)s * T + t];
      }
      davet_mailbox::Data* md = mailbox->dev;
      const int32_t stamp = (int32_t)(stamp0 + (uint32_t)t);
      rc = launch_policy_step(n_seqs, L, K, alpha.data(), lo_t.data(),
                              up_t.data(), conf, am, am_prev, resp_masked,
                              md->level, md->budget, nullptr, nullptr, nullptr,
                              &md->done, stamp, stream);
      if (rc) return rc;
      rc = wait_stamp(&mailbox->host->done, stamp, stream);
      if (rc) return rc;
    }
  }
  return DAVET_OK;
}
