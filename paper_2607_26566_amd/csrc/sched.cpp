// vTime fair scheduler (Sec. 6, Alg. 1): host-side control-plane library.
// Ready invocations are kept in submission order; tenants in an ordered map,
// so every decision is a deterministic function of the call sequence.
#include <cmath>
#include <map>
#include <new>
#include <unordered_map>
#include <vector>

#include "../../include/t2i_sched.h"

namespace {

struct Inv {
  int64_t id;
  int32_t tenant;
  double est, remaining, ready_at;
};

struct Tenant {
  double v = 0.0;
  bool active = false;
  int ready = 0, running = 0;
};

}  // namespace

struct t2i_sched {
  double delta;
  std::map<int32_t, Tenant> tenants;
  std::vector<Inv> ready;
  std::unordered_map<int64_t, Inv> running;
};

extern "C" {

t2i_status t2i_sched_create(double delta, t2i_sched** out) {
  if (!out) return T2I_ERR_INVALID_ARG;
  *out = nullptr;
  if (!(delta >= 0.0)) return T2I_ERR_INVALID_ARG;   // also rejects NaN
  t2i_sched* s = new (std::nothrow) t2i_sched();
  if (!s) return T2I_ERR_OUT_OF_MEMORY;
  s->delta = delta;
  *out = s;
  return T2I_OK;
}

void t2i_sched_destroy(t2i_sched* s) { delete s; }

t2i_status t2i_sched_submit(t2i_sched* s, int32_t tenant, int64_t fn_id, double est,
                            double remaining, double now) {
  if (!s) return T2I_ERR_INVALID_ARG;
  if (!(est > 0.0) || !std::isfinite(est) || !(remaining >= 0.0) || !std::isfinite(remaining) ||
      !std::isfinite(now))
    return T2I_ERR_INVALID_ARG;
  if (s->running.count(fn_id)) return T2I_ERR_INVALID_ARG;
  for (const Inv& n : s->ready)
    if (n.id == fn_id) return T2I_ERR_INVALID_ARG;
  s->ready.push_back({fn_id, tenant, est, remaining, now});
  s->tenants[tenant].ready++;
  return T2I_OK;
}

t2i_status t2i_sched_schedule(t2i_sched* s, double now, int32_t* picked, int64_t* fn_id,
                              int32_t* tenant, double* charged) {
  if (!s || !picked || !fn_id || !tenant || !charged || !std::isfinite(now))
    return T2I_ERR_INVALID_ARG;
  *picked = 0;
  if (s->ready.empty()) return T2I_OK;
  // vTime lift: tenants with ready work that are not active start at the
  // minimum vTime of the tenants active before this call
  bool any_active = false;
  double vact = 0.0;
  for (const auto& kv : s->tenants)
    if (kv.second.active) {
      vact = any_active ? std::fmin(vact, kv.second.v) : kv.second.v;
      any_active = true;
    }
  for (auto& kv : s->tenants) {
    Tenant& t = kv.second;
    if (t.ready > 0 && !t.active) {
      if (any_active) t.v = vact;
      t.active = true;
    }
  }
  // layer 1: candidates within delta of the smallest vTime with ready work
  bool first = true;
  double vmin = 0.0;
  for (const auto& kv : s->tenants)
    if (kv.second.ready > 0) {
      vmin = first ? kv.second.v : std::fmin(vmin, kv.second.v);
      first = false;
    }
  auto cand = [&](int32_t u) {
    const Tenant& t = s->tenants.at(u);
    return t.v - vmin <= s->delta;
  };
  // layer 2: normalised score over the candidates' ready invocations
  double wmax = 0.0, rmax = 0.0, emax = 0.0;
  bool any = false;
  for (const Inv& n : s->ready) {
    if (!cand(n.tenant)) continue;
    const double w = now - n.ready_at;
    wmax = any ? std::fmax(wmax, w) : w;
    rmax = any ? std::fmax(rmax, n.remaining) : n.remaining;
    emax = any ? std::fmax(emax, n.est) : n.est;
    any = true;
  }
  auto norm = [](double x, double m) { return m > 0.0 ? x / m : 0.0; };
  int best = -1;
  double best_s = 0.0;
  for (int i = 0; i < (int)s->ready.size(); ++i) {
    const Inv& n = s->ready[i];
    if (!cand(n.tenant)) continue;
    const double sc = norm(now - n.ready_at, wmax) - norm(n.remaining, rmax) - norm(n.est, emax);
    if (best < 0) {
      best = i;
      best_s = sc;
      continue;
    }
    const Inv& b = s->ready[best];
    if (sc > best_s || (sc == best_s && (n.ready_at < b.ready_at ||
                                         (n.ready_at == b.ready_at && n.id < b.id)))) {
      best = i;
      best_s = sc;
    }
  }
  const Inv n = s->ready[best];
  s->ready.erase(s->ready.begin() + best);
  Tenant& t = s->tenants[n.tenant];
  t.ready--;
  t.running++;
  t.v += n.est;
  s->running[n.id] = n;
  *picked = 1;
  *fn_id = n.id;
  *tenant = n.tenant;
  *charged = n.est;
  return T2I_OK;
}

t2i_status t2i_sched_complete(t2i_sched* s, int64_t fn_id, double measured) {
  if (!s || !std::isfinite(measured) || measured < 0.0) return T2I_ERR_INVALID_ARG;
  auto it = s->running.find(fn_id);
  if (it == s->running.end()) return T2I_ERR_INVALID_ARG;
  const Inv n = it->second;
  s->running.erase(it);
  Tenant& t = s->tenants[n.tenant];
  t.v += measured - n.est;
  t.running--;
  if (t.ready == 0 && t.running == 0) t.active = false;
  return T2I_OK;
}

t2i_status t2i_sched_vtime(const t2i_sched* s, int32_t tenant, double* v) {
  if (!s || !v) return T2I_ERR_INVALID_ARG;
  auto it = s->tenants.find(tenant);
  *v = it == s->tenants.end() ? 0.0 : it->second.v;
  return T2I_OK;
}

}  // extern "C"
