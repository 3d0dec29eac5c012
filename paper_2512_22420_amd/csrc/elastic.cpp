// Elastic KV pool control (Sec. 6.1-6.4): the trigger state machine and the
// draft weight offload / reload copies.  Host code; the transitions and their
// readings are listed in include/nightjar_memory.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/nightjar.h"
#include "../../include/nightjar_memory.h"
#include "kernels.h"

struct nj_elastic {
  nj_elastic_config cfg;
  int state = NJ_POOL_RESIDENT;
  int low = 0;   // consecutive steps with n_free < tau_low and no speculation
  int idle = 0;  // consecutive steps with no waiting request and n_free > n_draft + tau_low
  bool reload_pending = false;
};

extern "C" {

nj_elastic* nightjar_elastic_create(const nj_elastic_config* cfg) {
  if (!cfg || cfg->n_orig < 1 || cfg->n_draft < 0 || cfg->tau_low < 0 || cfg->t_persist < 1 ||
      cfg->reload_persist < 1 || cfg->max_migrate < 0) {
    nj::set_last_error(NJ_EINVAL, "elastic config: need n_orig >= 1, n_draft, tau_low, max_migrate >= 0, "
                                  "t_persist, reload_persist >= 1");
    return nullptr;
  }
  nj_elastic* e = new nj_elastic;
  e->cfg = *cfg;
  return e;
}

void nightjar_elastic_destroy(nj_elastic* e) { delete e; }

int nightjar_elastic_step(nj_elastic* e, int32_t n_free, int32_t n_waiting, int32_t speculating, int32_t live_above,
                          int32_t* action) {
  if (!e || !action) return nj::set_last_error(NJ_EINVAL, "elastic_step: NULL argument");
  if (n_free < 0 || n_waiting < 0 || live_above < 0) return nj::set_last_error(NJ_EINVAL, "elastic_step: negative count");
  const nj_elastic_config& c = e->cfg;
  e->low = (n_free < c.tau_low && !speculating) ? e->low + 1 : 0;
  e->idle = (n_waiting == 0 && n_free > c.n_draft + c.tau_low) ? e->idle + 1 : 0;
  int act = NJ_ACT_NONE;
  switch (e->state) {
    case NJ_POOL_RESIDENT:
      if (e->low >= c.t_persist) {
        act = NJ_ACT_OFFLOAD_DRAFT;
        e->state = NJ_POOL_OFFLOADING;
      }
      break;
    case NJ_POOL_OFFLOADED:
      if (e->reload_pending) {
        act = NJ_ACT_RELOAD_DRAFT;
        e->state = NJ_POOL_RELOADING;
        e->reload_pending = false;
      } else if (e->low >= c.t_persist) {
        act = NJ_ACT_EXPAND;
        e->state = NJ_POOL_EXPANDED;
      } else if (e->idle >= c.reload_persist) {
        act = NJ_ACT_RELOAD_DRAFT;
        e->state = NJ_POOL_RELOADING;
      }
      break;
    case NJ_POOL_EXPANDED:
      if (e->idle >= c.reload_persist && live_above <= c.max_migrate) {
        act = NJ_ACT_CONTRACT;
        e->state = NJ_POOL_CONTRACTING;
      }
      break;
    default:  // an asynchronous action is in flight
      break;
  }
  *action = act;
  return NJ_OK;
}

int nightjar_elastic_done(nj_elastic* e, int32_t action) {
  if (!e) return nj::set_last_error(NJ_EINVAL, "elastic_done: NULL");
  if (action == NJ_ACT_OFFLOAD_DRAFT && e->state == NJ_POOL_OFFLOADING) {
    e->state = NJ_POOL_OFFLOADED;
  } else if (action == NJ_ACT_CONTRACT && e->state == NJ_POOL_CONTRACTING) {
    e->state = NJ_POOL_OFFLOADED;
    e->reload_pending = true;  // the draft comes back once the pool is shrunk
  } else if (action == NJ_ACT_RELOAD_DRAFT && e->state == NJ_POOL_RELOADING) {
    e->state = NJ_POOL_RESIDENT;
  } else {
    return nj::set_last_error(NJ_EINVAL, "elastic_done: action %d is not in flight (state %d)", action, e->state);
  }
  return NJ_OK;
}

int nightjar_elastic_state(const nj_elastic* e, int32_t* state, int32_t* pool_blocks, int32_t* gamma_allowed) {
  if (!e || !state || !pool_blocks || !gamma_allowed) return nj::set_last_error(NJ_EINVAL, "elastic_state: NULL");
  *state = e->state;
  const bool big = e->state == NJ_POOL_EXPANDED || e->state == NJ_POOL_CONTRACTING;
  *pool_blocks = e->cfg.n_orig + (big ? e->cfg.n_draft : 0);
  *gamma_allowed = e->state == NJ_POOL_RESIDENT;
  return NJ_OK;
}

int nightjar_offload(const void* device_src, void* host_dst, size_t bytes, void* stream) {
  if (!device_src || !host_dst) return nj::set_last_error(NJ_EINVAL, "offload: NULL pointer");
  const hipError_t e = hipMemcpyAsync(host_dst, device_src, bytes, hipMemcpyDeviceToHost, (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : nj::set_last_error(NJ_EHIP, "offload: %s", hipGetErrorString(e));
}

int nightjar_reload(const void* host_src, void* device_dst, size_t bytes, void* stream) {
  if (!host_src || !device_dst) return nj::set_last_error(NJ_EINVAL, "reload: NULL pointer");
  const hipError_t e = hipMemcpyAsync(device_dst, host_src, bytes, hipMemcpyHostToDevice, (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : nj::set_last_error(NJ_EHIP, "reload: %s", hipGetErrorString(e));
}

}  // extern "C"
