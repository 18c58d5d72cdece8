// C ABI of the SpecTrain stage library: argument checks, status codes and the
// thread-local error message. No exception crosses this boundary.
#include <new>
#include <string>

#include "stage.hpp"

struct spectrain_stage {
  spx::Stage* impl;
};

namespace {

thread_local std::string g_last_error;

int set_error(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

template <typename F>
int guarded(spectrain_stage_t st, F&& f, bool check_flag = true) {
  if (!st || !st->impl) return set_error(SPECTRAIN_EINVAL, "stage handle is NULL");
  try {
    if (check_flag && st->impl->nonfinite())
      return set_error(SPECTRAIN_ENONFINITE, "an update produced a non-finite weight or smoothed gradient");
    f(*st->impl);
    g_last_error.clear();
    return SPECTRAIN_OK;
  } catch (const spx::StageError& e) {
    return set_error(e.code, e.what());
  } catch (const std::bad_alloc&) {
    return set_error(SPECTRAIN_ENOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    return set_error(SPECTRAIN_EINVAL, e.what());
  } catch (...) {
    return set_error(SPECTRAIN_EINVAL, "unknown failure");
  }
}

}  // namespace

extern "C" {

int32_t spectrain_version_difference(int32_t k, int32_t N, int32_t is_forward) {
  if (N < 1 || k < 0 || k >= N) return -1;
  return is_forward ? k / 2 + N - k - 1 : k / 2;   // Eq. 5 / Eq. 6
}

int spectrain_stage_create(const spectrain_stage_desc* desc, const float* W0_host, size_t n_params, void* hip_stream,
                           spectrain_stage_t* out) {
  if (!desc || !out) return set_error(SPECTRAIN_EINVAL, "desc and out must not be NULL");
  *out = nullptr;
  spectrain_stage* h = nullptr;
  try {
    h = new spectrain_stage{nullptr};
    h->impl = new spx::Stage(*desc, W0_host, n_params, static_cast<hipStream_t>(hip_stream));
    *out = h;
    g_last_error.clear();
    return SPECTRAIN_OK;
  } catch (const spx::StageError& e) {
    delete h;
    return set_error(e.code, e.what());
  } catch (const std::bad_alloc&) {
    delete h;
    return set_error(SPECTRAIN_ENOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    delete h;
    return set_error(SPECTRAIN_EINVAL, e.what());
  }
}

int spectrain_stage_num_params(spectrain_stage_t st, size_t* n) {
  if (!n) return set_error(SPECTRAIN_EINVAL, "n is NULL");
  return guarded(st, [&](spx::Stage& s) { *n = s.num_params(); }, false);
}

int spectrain_stage_predict(spectrain_stage_t st, int32_t s, int32_t slot) {
  return guarded(st, [&](spx::Stage& x) { x.predict(s, slot); });
}

int spectrain_stage_forward(spectrain_stage_t st, int64_t mb_id, const void* x_dev, void* y_dev,
                            const int32_t* labels_dev, float* loss_dev) {
  return guarded(st, [&](spx::Stage& x) { x.forward(mb_id, x_dev, y_dev, labels_dev, loss_dev); });
}

int spectrain_stage_backward(spectrain_stage_t st, int64_t mb_id, const void* dy_dev, void* dx_dev) {
  return guarded(st, [&](spx::Stage& x) { x.backward(mb_id, dy_dev, dx_dev); });
}

int spectrain_stage_backward_noalloc(spectrain_stage_t st, int64_t mb_id, const void* dy_dev, void* dx_dev) {
  return guarded(st, [&](spx::Stage& x) { x.backward_noalloc(mb_id, dy_dev, dx_dev); });
}

int spectrain_stage_forward_backward(spectrain_stage_t st, int64_t mb_fwd, const void* x_dev, void* y_dev,
                                     const int32_t* labels_dev, float* loss_dev, int64_t mb_bwd, const void* dy_dev,
                                     void* dx_dev) {
  return guarded(st, [&](spx::Stage& x) {
    x.forward_backward(mb_fwd, x_dev, y_dev, labels_dev, loss_dev, mb_bwd, dy_dev, dx_dev);
  });
}

int spectrain_stage_update(spectrain_stage_t st, int32_t s_next_fwd, int32_t s_next_bwd) {
  return guarded(st, [&](spx::Stage& x) { x.update(s_next_fwd, s_next_bwd); });
}

int spectrain_stage_get_state(spectrain_stage_t st, float* W_host, float* v_host) {
  return guarded(st, [&](spx::Stage& x) { x.get_state(W_host, v_host); }, false);
}

int spectrain_stage_set_state(spectrain_stage_t st, const float* W_host, const float* v_host) {
  return guarded(st, [&](spx::Stage& x) { x.set_state(W_host, v_host); }, false);
}

int spectrain_stage_get_predicted(spectrain_stage_t st, int32_t slot, float* What_host) {
  return guarded(st, [&](spx::Stage& x) { x.get_predicted(slot, What_host); }, false);
}

int spectrain_stage_read_stash(spectrain_stage_t st, int64_t mb_id, int32_t index, void* host_out, size_t capacity,
                               size_t* size) {
  if (!size) return set_error(SPECTRAIN_EINVAL, "size is NULL");
  return guarded(st, [&](spx::Stage& x) { *size = x.read_stash(mb_id, index, host_out, capacity); }, false);
}

int spectrain_stage_profile(spectrain_stage_t st, int32_t enable) {
  return guarded(st, [&](spx::Stage& x) {
    if (enable < 0 || enable > 2) throw spx::StageError(SPECTRAIN_EINVAL, "profile mode must be 0, 1 or 2");
    x.profile(enable != 0, enable == 2);
  }, false);
}

int spectrain_stage_profile_read(spectrain_stage_t st, spectrain_kernel_stat* out, int32_t capacity, int32_t* count) {
  if (!count || (capacity > 0 && !out)) return set_error(SPECTRAIN_EINVAL, "out and count must not be NULL");
  return guarded(st, [&](spx::Stage& x) { *count = x.profile_read(out, capacity); }, false);
}

int spectrain_stage_destroy(spectrain_stage_t st) {
  if (!st) return set_error(SPECTRAIN_EINVAL, "stage handle is NULL");
  delete st->impl;
  delete st;
  g_last_error.clear();
  return SPECTRAIN_OK;
}

const char* spectrain_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
