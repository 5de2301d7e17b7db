// controller.cpp -- the TempoKV claim / commitment controller (Section 3)
// driven by a discrete-event model of the serving runtime and the staging
// device.  Host code; no GPU calls.
//
// Claims are reported PLANNED when their request arrives.  At every control
// point (after each event and every tick) the controller first admits
// waiting requests to free runtime slots (an admitted request requests the
// retrieval of its claim), then walks the PLANNED claims -- those with a
// pending retrieval request first, then the waiting ones in the runtime's
// FCFS order (Section 3.2 "Commitment and replanning") -- and asks the
// commitment rule kv_commit_should_stage for each: eligibility from the
// policy (or the retrieval request), capacity from the protected budget.  A
// claim that cannot commit holds up no later claim; a commitment is never revoked; a
// claim that cannot be protected when its retrieval is requested takes the
// ordinary path (Section 3.2 "Protected capacity and on-demand retrieval").
//
// Commitment protects each object of the claim's manifest and queues a
// staging read for every one neither resident nor already being staged, so
// shared objects are read and reserved once (Section 3.2 "Shared staging and
// resource lifecycle").  The claim is STAGEREADY once all its objects are
// resident, TRANSFERRING when retrieval begins, RELEASED when it ends.
//
// TTU (Section 3.1, "Runtime-estimated time-to-use") projects the FCFS slots
// assuming the target and the requests ahead are stage-ready.  TTR: static
// (non-resident bytes over a fixed rate, the claim in isolation) or
// state-aware (the staging queue projected: queued objects keep their
// completion times, new reads are appended; the last object decides).
//
// The arithmetic follows one fixed order so that runs are reproducible and
// comparable event by event; the file is compiled without floating-point
// contraction.

#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <functional>
#include <queue>
#include <tuple>
#include <vector>

#include "tempokv.h"

namespace {

// TTR estimators (Section 3.1, "Storage-estimated time-to-ready") over a
// claim's distinct KV objects; shared by the simulator and the C ABI.
// Static: the non-resident bytes over a fixed rate, the claim in isolation.
template <class Flag>
double ttr_static_of(const int32_t *objs, size_t n, const double *bytes, const Flag *resident, double rate) {
    double s = 0.0;
    for (size_t k = 0; k < n; ++k)
        if (!resident[objs[k]]) s += bytes[objs[k]];
    return s / rate;
}

// State-aware: the staging queue projected from `now`.  An object already
// queued keeps its completion time; a non-resident object not yet queued is
// appended behind the queue's tail (busy until `busy_until`) at the staging
// rate; the last object to become resident decides.
template <class Flag>
double ttr_state_of(const int32_t *objs, size_t n, const double *bytes, const Flag *resident, const Flag *queued,
                    const double *ready_at, double now, double busy_until, double stage_rate) {
    double t_end = now;
    double tail = std::max(busy_until, now);
    for (size_t k = 0; k < n; ++k) {
        const int32_t o = objs[k];
        if (resident[o]) continue;
        if (queued[o]) {
            t_end = std::max(t_end, ready_at[o]);
        } else {
            tail = tail + bytes[o] / stage_rate;
            t_end = std::max(t_end, tail);
        }
    }
    return t_end - now;
}

enum { PLANNED, STAGING, STAGEREADY, TRANSFERRING, RELEASED, ORDINARY };
enum { EV_ARRIVAL, EV_OBJ_READY, EV_FETCH_END, EV_TRANSFER_END, EV_REQ_END, EV_TICK };
enum { PH_WAIT, PH_FETCH, PH_RUN };

struct Event {
    double t;
    int64_t seq;
    int kind;
    int32_t a;
    bool operator>(const Event &o) const { return t > o.t || (t == o.t && seq > o.seq); }
};

class Sim {
  public:
    Sim(const kv_sim_config &c, const double *obj_bytes, int32_t O, const double *arrival, const int64_t *moff,
        const int32_t *mobj, const int32_t *unc, const int32_t *out, int32_t N, kv_sim_event *trace, int64_t cap)
        : c_(c), bytes_(obj_bytes, obj_bytes + O), arrival_(arrival, arrival + N), unc_(unc, unc + N),
          out_(out, out + N), N_(N), O_(O), trace_(trace), trace_cap_(cap) {
        resident_.assign(O, 0);
        queued_.assign(O, 0);
        ready_at_.assign(O, 0.0);
        prot_.assign(O, 0);
        lru_.assign(O, 0.0);
        uniq_.resize(N);
        std::vector<int64_t> seen(O, -1);
        for (int32_t i = 0; i < N; ++i)
            for (int64_t k = moff[i]; k < moff[i + 1]; ++k) {
                const int32_t o = mobj[k];
                if (seen[o] != i) {
                    seen[o] = i;
                    uniq_[i].push_back(o);
                }
            }
        total_.assign(N, 0.0);
        svc_.assign(N, 0.0);
        for (int32_t i = 0; i < N; ++i) {
            double s = 0.0;
            for (int32_t o : uniq_[i]) s += bytes_[o];
            total_[i] = s;
            svc_[i] = total_[i] / c_.gpu_rate + (double)unc_[i] * c_.prefill_s + (double)out_[i] * c_.decode_s;
        }
        state_.assign(N, PLANNED);
        requested_.assign(N, 0);
        blocked_.assign(N, 0);
        phase_.assign(N, PH_WAIT);
        fetch_end_.assign(N, 0.0);
        req_end_.assign(N, 0.0);
        first_token_.assign(N, NAN);
        done_.assign(N, NAN);
    }

    void run(kv_sim_result *res) {
        for (int32_t i = 0; i < N_; ++i) push(arrival_[i], EV_ARRIVAL, i);
        push(0.0, EV_TICK, 0);
        int32_t n_done = 0;
        int64_t nev = 0;
        while (!heap_.empty() && n_done < N_) {
            const Event e = heap_.top();
            heap_.pop();
            ++nev;
            area_ += P_ * (e.t - now_);
            now_ = e.t;
            switch (e.kind) {
            case EV_ARRIVAL:
                waiting_.push_back(e.a);
                tr(KV_TR_ARRIVE, e.a);
                break;
            case EV_OBJ_READY:
                queued_[e.a] = 0;
                make_resident(e.a, true);
                tr(KV_TR_READY, e.a);
                for (int32_t i = 0; i < N_; ++i)
                    if (state_[i] == STAGING && all_resident(i)) {
                        state_[i] = STAGEREADY;
                        tr(KV_TR_STAGEREADY, i);
                    }
                break;
            case EV_FETCH_END:
                for (int32_t o : uniq_[e.a])
                    if (!resident_[o]) make_resident(o, false);
                start_run(e.a);
                break;
            case EV_TRANSFER_END:
                if (state_[e.a] == TRANSFERRING) {
                    state_[e.a] = RELEASED;
                    for (int32_t o : uniq_[e.a]) {
                        if (--prot_[o] == 0) {
                            P_ -= bytes_[o];
                            lru_[o] = now_;
                        }
                    }
                    tr(KV_TR_RELEASE, e.a);
                }
                break;
            case EV_REQ_END:
                done_[e.a] = now_;
                active_.erase(std::find(active_.begin(), active_.end(), e.a));
                ++n_done;
                tr(KV_TR_DONE, e.a);
                break;
            case EV_TICK:
                push((double)(e.a + 1) * c_.tick_s, EV_TICK, e.a + 1);
                break;
            }
            control();
        }
        res->area_byte_s = area_;
        res->cost_gib_s_per_request = N_ ? area_ / 1073741824.0 / (double)N_ : 0.0;
        res->end_s = now_;
        res->p_max_bytes = P_max_;
        res->committed = committed_;
        int32_t nb = 0, no = 0;
        for (int32_t i = 0; i < N_; ++i) {
            nb += blocked_[i] ? 1 : 0;
            no += state_[i] == ORDINARY ? 1 : 0;
        }
        res->blocked = nb;
        res->ordinary = no;
        res->reserved = 0;
        res->events = nev;
    }

    const std::vector<double> &first_token() const { return first_token_; }
    const std::vector<double> &done() const { return done_; }
    int64_t trace_len() const { return trace_len_; }

  private:
    void push(double t, int kind, int32_t a) { heap_.push(Event{t, seq_++, kind, a}); }

    void tr(int kind, int32_t id) {
        if (trace_ && trace_len_ < trace_cap_) trace_[trace_len_] = kv_sim_event{now_, kind, id};
        ++trace_len_;
    }

    bool all_resident(int32_t i) const {
        for (int32_t o : uniq_[i])
            if (!resident_[o]) return false;
        return true;
    }

    // An object becomes resident; least-recently-released unprotected objects
    // (ties by id) are evicted until it fits.  A protected object always fits
    // (protected bytes <= budget <= capacity); an unprotected one that does
    // not is not retained.
    void make_resident(int32_t o, bool is_protected) {
        if (resident_[o]) {
            lru_[o] = now_;
            return;
        }
        if (used_ + bytes_[o] > c_.capacity_bytes) {
            std::vector<int32_t> victims;
            for (int32_t x = 0; x < O_; ++x)
                if (resident_[x] && prot_[x] == 0 && x != o) victims.push_back(x);
            std::sort(victims.begin(), victims.end(), [&](int32_t a, int32_t b) {
                return lru_[a] < lru_[b] || (lru_[a] == lru_[b] && a < b);
            });
            for (int32_t x : victims) {
                if (used_ + bytes_[o] <= c_.capacity_bytes) break;
                resident_[x] = 0;
                used_ -= bytes_[x];
                tr(KV_TR_EVICT, x);
            }
        }
        if (used_ + bytes_[o] <= c_.capacity_bytes || is_protected) {
            resident_[o] = 1;
            used_ += bytes_[o];
            lru_[o] = now_;
        }
    }

    double ttr_static(int32_t i) const {
        return ttr_static_of(uniq_[i].data(), uniq_[i].size(), bytes_.data(), resident_.data(), c_.static_rate);
    }

    double ttr_state(int32_t i) const {
        return ttr_state_of(uniq_[i].data(), uniq_[i].size(), bytes_.data(), resident_.data(), queued_.data(),
                            ready_at_.data(), now_, busy_until_, c_.stage_rate);
    }

    double projected_end(int32_t i) const {
        if (phase_[i] == PH_RUN) return req_end_[i];
        if (phase_[i] == PH_FETCH) return fetch_end_[i] + svc_[i];
        if (state_[i] == STAGING) {
            double r = now_;
            for (int32_t o : uniq_[i])
                if (!resident_[o] && queued_[o]) r = std::max(r, ready_at_[o]);
            return r + svc_[i];
        }
        return now_ + svc_[i];
    }

    // TTU of every waiting request, in the waiting order.
    void ttus(std::vector<double> &out) const {
        std::priority_queue<double, std::vector<double>, std::greater<double>> slots;
        for (int32_t a : active_) slots.push(projected_end(a));
        for (size_t k = active_.size(); k < (size_t)c_.max_active; ++k) slots.push(now_);
        out.assign(N_, INFINITY);
        for (int32_t w : waiting_) {
            const double s0 = std::max(slots.top(), now_);
            out[w] = s0 - now_;
            slots.pop();
            slots.push(s0 + svc_[w]);
        }
    }

    void commit(int32_t i) {
        for (int32_t o : uniq_[i]) {
            if (prot_[o] == 0) {
                P_ += bytes_[o];
                P_max_ = std::max(P_max_, P_);
            }
            prot_[o] += 1;
            if (!resident_[o] && !queued_[o]) {
                const double start = std::max(now_, busy_until_);
                ready_at_[o] = start + bytes_[o] / c_.stage_rate;
                busy_until_ = ready_at_[o];
                queued_[o] = 1;
                push(ready_at_[o], EV_OBJ_READY, o);
            }
        }
        state_[i] = all_resident(i) ? STAGEREADY : STAGING;
        ++committed_;
        tr(KV_TR_COMMIT, i);
    }

    int decide(int32_t i, int64_t pos, const std::vector<double> &ttu) const {
        double nw = 0.0;
        for (int32_t o : uniq_[i])
            if (prot_[o] == 0) nw += bytes_[o];
        double t_u = 0.0, t_r = 0.0;
        switch (c_.policy) {
        case KV_POLICY_DEMAND: t_u = INFINITY; break;
        case KV_POLICY_IMMEDIATE: t_u = -INFINITY; break;
        case KV_POLICY_QUEUE_K: t_u = (pos >= 0 && pos < c_.queue_k) ? -INFINITY : INFINITY; break;
        case KV_POLICY_TEMPO_STATIC: t_u = ttu[i]; t_r = ttr_static(i); break;
        default: t_u = ttu[i]; t_r = ttr_state(i); break;
        }
        return kv_commit_should_stage(t_u, t_r, (uint64_t)(c_.budget_bytes - P_), (uint64_t)nw, (uint64_t)total_[i],
                                      (uint64_t)c_.budget_bytes, requested_[i]);
    }

    void start_run(int32_t i) {
        phase_[i] = PH_RUN;
        const double t_x = now_ + total_[i] / c_.gpu_rate;
        first_token_[i] = t_x + (double)unc_[i] * c_.prefill_s;
        req_end_[i] = first_token_[i] + (double)out_[i] * c_.decode_s;
        push(t_x, EV_TRANSFER_END, i);
        push(req_end_[i], EV_REQ_END, i);
    }

    void control() {
        while (!waiting_.empty() && (int32_t)active_.size() < c_.max_active) {
            const int32_t i = waiting_.front();
            waiting_.erase(waiting_.begin());
            active_.push_back(i);
            requested_[i] = 1;
            phase_[i] = PH_WAIT;
            tr(KV_TR_ADMIT, i);
        }
        std::vector<int32_t> order;
        for (int32_t i : active_)
            if (state_[i] == PLANNED) order.push_back(i);
        for (int32_t i : waiting_)
            if (state_[i] == PLANNED) order.push_back(i);
        const bool tempo = c_.policy == KV_POLICY_TEMPO || c_.policy == KV_POLICY_TEMPO_STATIC;
        std::vector<double> ttu;
        if (tempo) ttus(ttu);
        else ttu.assign(N_, INFINITY);
        std::vector<int64_t> pos(N_, -1);
        for (size_t k = 0; k < waiting_.size(); ++k) pos[waiting_[k]] = (int64_t)k;
        for (int32_t i : order) {
            const int d = decide(i, pos[i], ttu);
            if (d == KV_COMMIT) {
                commit(i);
                if (tempo) ttus(ttu);
            } else if (d == KV_ORDINARY) {
                state_[i] = ORDINARY;
                tr(KV_TR_ORDINARY, i);
            } else if (d == KV_BLOCKED) {
                blocked_[i] = 1;
            }
        }
        const std::vector<int32_t> act = active_;
        for (int32_t i : act) {
            if (phase_[i] != PH_WAIT) continue;
            if (state_[i] == STAGEREADY) {
                state_[i] = TRANSFERRING;
                start_run(i);
                tr(KV_TR_TRANSFER, i);
            } else if (state_[i] == ORDINARY) {
                phase_[i] = PH_FETCH;
                double nonres = 0.0;
                for (int32_t o : uniq_[i])
                    if (!resident_[o]) nonres += bytes_[o];
                fetch_end_[i] = std::max(now_, busy_until_) + nonres / c_.stage_rate;
                busy_until_ = fetch_end_[i];
                push(fetch_end_[i], EV_FETCH_END, i);
                tr(KV_TR_FETCH, i);
            }
        }
    }

    const kv_sim_config c_;
    const std::vector<double> bytes_, arrival_;
    const std::vector<int32_t> unc_, out_;
    const int32_t N_, O_;
    kv_sim_event *trace_;
    const int64_t trace_cap_;
    int64_t trace_len_ = 0;

    std::vector<char> resident_, queued_;
    std::vector<double> ready_at_, lru_;
    std::vector<int32_t> prot_;
    std::vector<std::vector<int32_t>> uniq_;
    std::vector<double> total_, svc_;
    std::vector<int> state_, phase_;
    std::vector<char> requested_, blocked_;
    std::vector<double> fetch_end_, req_end_, first_token_, done_;
    std::vector<int32_t> waiting_, active_;
    std::priority_queue<Event, std::vector<Event>, std::greater<Event>> heap_;
    int64_t seq_ = 0;
    double now_ = 0.0, P_ = 0.0, P_max_ = 0.0, area_ = 0.0, busy_until_ = 0.0, used_ = 0.0;
    int32_t committed_ = 0;
};

}  // namespace

extern "C" int kv_sim_run(const kv_sim_config *cfg, const double *h_obj_bytes, int32_t num_objects,
                          const double *h_arrival, const int64_t *h_manifest_off, const int32_t *h_manifest_objs,
                          const int32_t *h_uncached, const int32_t *h_out_tokens, int32_t num_requests,
                          double *h_first_token, double *h_done, kv_sim_result *result, kv_sim_event *h_trace,
                          int64_t trace_cap, int64_t *trace_len) {
    if (!cfg || !result || num_objects < 0 || num_requests < 0 || trace_cap < 0) return KV_EINVAL;
    if (num_requests > 0 && (!h_arrival || !h_manifest_off || !h_uncached || !h_out_tokens || !h_first_token ||
                             !h_done))
        return KV_EINVAL;
    if (num_objects > 0 && !h_obj_bytes) return KV_EINVAL;
    if (cfg->reserved != 0 || cfg->max_active <= 0 || cfg->queue_k < 0 || cfg->policy < 0 ||
        cfg->policy > KV_POLICY_TEMPO)
        return KV_EINVAL;
    if (!(cfg->budget_bytes >= 0) || !(cfg->capacity_bytes >= cfg->budget_bytes) || !(cfg->stage_rate > 0) ||
        !(cfg->static_rate > 0) || !(cfg->gpu_rate > 0) || !(cfg->prefill_s >= 0) || !(cfg->decode_s >= 0) ||
        !(cfg->tick_s > 0))
        return KV_EINVAL;
    for (int32_t o = 0; o < num_objects; ++o)
        if (!(h_obj_bytes[o] >= 0) || h_obj_bytes[o] > 9007199254740992.0 || h_obj_bytes[o] != floor(h_obj_bytes[o]))
            return KV_EINVAL;
    if (num_requests > 0) {
        if (h_manifest_off[0] != 0) return KV_EINVAL;
        for (int32_t i = 0; i < num_requests; ++i) {
            if (h_manifest_off[i + 1] < h_manifest_off[i] || !(h_arrival[i] >= 0) || h_uncached[i] < 0 ||
                h_out_tokens[i] < 0)
                return KV_EINVAL;
        }
        if (h_manifest_off[num_requests] > 0 && !h_manifest_objs) return KV_EINVAL;
        for (int64_t k = 0; k < h_manifest_off[num_requests]; ++k)
            if (h_manifest_objs[k] < 0 || h_manifest_objs[k] >= num_objects) return KV_EINVAL;
    }
    Sim sim(*cfg, h_obj_bytes, num_objects, h_arrival, h_manifest_off, h_manifest_objs, h_uncached, h_out_tokens,
            num_requests, h_trace, trace_cap);
    sim.run(result);
    for (int32_t i = 0; i < num_requests; ++i) {
        h_first_token[i] = sim.first_token()[i];
        h_done[i] = sim.done()[i];
    }
    if (trace_len) *trace_len = sim.trace_len();
    return KV_OK;
}

namespace {

// Objects of a claim: non-negative ids below num_objects.
bool objs_ok(int32_t n, const int32_t *objs, int32_t num_objects) {
    for (int32_t k = 0; k < n; ++k)
        if (objs[k] < 0 || objs[k] >= num_objects) return false;
    return true;
}

}  // namespace

extern "C" int kv_ttr_static(int32_t num_objs, const int32_t *h_objs, int32_t num_objects, const double *h_obj_bytes,
                             const uint8_t *h_resident, double static_rate, double *ttr_s) {
    if (num_objs < 0 || num_objects < 0 || !ttr_s || !(static_rate > 0)) return KV_EINVAL;
    if (num_objs > 0 && (!h_objs || !h_obj_bytes || !h_resident || !objs_ok(num_objs, h_objs, num_objects)))
        return KV_EINVAL;
    *ttr_s = ttr_static_of(h_objs, (size_t)num_objs, h_obj_bytes, h_resident, static_rate);
    return KV_OK;
}

extern "C" int kv_ttr_state_aware(int32_t num_objs, const int32_t *h_objs, int32_t num_objects,
                                  const double *h_obj_bytes, const uint8_t *h_resident, const uint8_t *h_queued,
                                  const double *h_ready_at, double now_s, double busy_until_s, double stage_rate,
                                  double *ttr_s) {
    if (num_objs < 0 || num_objects < 0 || !ttr_s || !(stage_rate > 0) || isnan(now_s) || isnan(busy_until_s))
        return KV_EINVAL;
    if (num_objs > 0 && (!h_objs || !h_obj_bytes || !h_resident || !h_queued || !h_ready_at ||
                         !objs_ok(num_objs, h_objs, num_objects)))
        return KV_EINVAL;
    *ttr_s = ttr_state_of(h_objs, (size_t)num_objs, h_obj_bytes, h_resident, h_queued, h_ready_at, now_s,
                          busy_until_s, stage_rate);
    return KV_OK;
}
