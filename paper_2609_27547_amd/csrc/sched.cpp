// Rollout scheduler feeding the generation calls: group pipeline between
// simulation and generation (Section 4.2.2) and greedy core rebinding
// (Section 4.2.3, Algorithm 2, ready set of Eq. (1)).  Host-only C++; the
// model and its readings are stated in ebrl_sched.h.
#include <stdint.h>

#include <deque>
#include <mutex>
#include <new>
#include <vector>

#include "ebrl.h"
#include "ebrl_sched.h"

namespace {
enum GroupState { QUEUED, GENERATING, ACTIVE };
}

struct ebrl_sched {
    int32_t n_envs, n_groups, K;
    std::vector<int32_t> done;        // s_e: actions done in the current chunk
    std::vector<uint8_t> running;     // step in flight
    std::vector<uint8_t> has_chunk;   // a chunk was delivered (actions available while done < K)
    std::vector<double> last;         // H[e]: most recent step duration, < 0 = none recorded
    std::vector<int32_t> left;        // per group: envs that have not finished the chunk
    std::vector<uint8_t> gstate;
    std::deque<int32_t> queue;        // groups waiting for generation, in completion order
    mutable std::mutex mu;

    std::vector<int32_t> group;       // env -> group
    int32_t first(int32_t g) const { return (int32_t)((int64_t)g * n_envs / n_groups); }
};

extern "C" {

int ebrl_sched_create(int32_t n_envs, int32_t n_groups, int32_t chunk_len, ebrl_sched** out) {
    if (!out || n_groups < 1 || n_groups > n_envs || chunk_len < 1) return EBRL_E_INVALID;
    ebrl_sched* s = new (std::nothrow) ebrl_sched;
    if (!s) return EBRL_E_OOM;
    s->n_envs = n_envs;
    s->n_groups = n_groups;
    s->K = chunk_len;
    s->done.assign(n_envs, 0);
    s->running.assign(n_envs, 0);
    s->has_chunk.assign(n_envs, 0);
    s->last.assign(n_envs, -1.0);
    s->left.assign(n_groups, 0);
    s->gstate.assign(n_groups, QUEUED);
    s->group.assign(n_envs, 0);
    for (int32_t g = 0; g < n_groups; ++g) {
        for (int32_t e = s->first(g); e < s->first(g + 1); ++e) s->group[e] = g;
        s->queue.push_back(g);
    }
    *out = s;
    return EBRL_OK;
}

void ebrl_sched_destroy(ebrl_sched* s) { delete s; }

int ebrl_sched_dispatch(ebrl_sched* s, int32_t core, int32_t bind_stride, int32_t* env) {
    if (!s || !env || bind_stride < 0 || (bind_stride > 0 && (core < 0 || core >= bind_stride)))
        return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(s->mu);
    int32_t pick = -1;
    for (int32_t e = bind_stride ? core : 0; e < s->n_envs; e += bind_stride ? bind_stride : 1) {
        if (!s->has_chunk[e] || s->running[e] || s->done[e] >= s->K) continue;   // Eq. (1)
        if (pick < 0) { pick = e; continue; }
        const double h = s->last[e], hp = s->last[pick];
        // no recorded step beats any recorded one; then the longer duration
        const bool better = (h < 0 && hp >= 0) || (h >= 0 && hp >= 0 && h > hp);
        if (better) pick = e;
    }
    if (pick >= 0) s->running[pick] = 1;
    *env = pick;
    return EBRL_OK;
}

int ebrl_sched_complete(ebrl_sched* s, int32_t env, double duration, int32_t* group_done) {
    if (!s || !group_done || env < 0 || !(duration >= 0)) return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(s->mu);
    if (env >= s->n_envs) return EBRL_E_INVALID;
    if (!s->running[env]) return EBRL_E_STATE;
    s->running[env] = 0;
    s->done[env] += 1;
    s->last[env] = duration;
    *group_done = 0;
    if (s->done[env] == s->K) {
        const int32_t g = s->group[env];
        if (--s->left[g] == 0) {
            for (int32_t e = s->first(g); e < s->first(g + 1); ++e) s->has_chunk[e] = 0;
            s->gstate[g] = QUEUED;
            s->queue.push_back(g);
            *group_done = 1;
        }
    }
    return EBRL_OK;
}

int ebrl_sched_next_group(ebrl_sched* s, int32_t* group, int32_t* env_ids, int32_t cap, int32_t* n) {
    if (!s || !group || !n) return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(s->mu);
    *group = -1;
    *n = 0;
    if (s->queue.empty()) return EBRL_OK;
    const int32_t g = s->queue.front();
    const int32_t a = s->first(g), b = s->first(g + 1);
    if (!env_ids || cap < b - a) return EBRL_E_INVALID;
    s->queue.pop_front();
    s->gstate[g] = GENERATING;
    for (int32_t e = a; e < b; ++e) env_ids[e - a] = e;
    *group = g;
    *n = b - a;
    return EBRL_OK;
}

int ebrl_sched_deliver(ebrl_sched* s, int32_t group) {
    if (!s) return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(s->mu);
    if (group < 0 || group >= s->n_groups) return EBRL_E_INVALID;
    if (s->gstate[group] != GENERATING) return EBRL_E_STATE;
    const int32_t a = s->first(group), b = s->first(group + 1);
    for (int32_t e = a; e < b; ++e) {
        s->done[e] = 0;
        s->has_chunk[e] = 1;
    }
    s->left[group] = b - a;
    s->gstate[group] = ACTIVE;
    return EBRL_OK;
}

int ebrl_sched_env_state(const ebrl_sched* s, int32_t env, int32_t* steps_done, int32_t* running,
                         int32_t* has_chunk, double* last_duration) {
    if (!s || env < 0 || env >= s->n_envs || !steps_done || !running || !has_chunk || !last_duration)
        return EBRL_E_INVALID;
    std::lock_guard<std::mutex> lk(s->mu);
    *steps_done = s->done[env];
    *running = s->running[env];
    *has_chunk = s->has_chunk[env];
    *last_duration = s->last[env];
    return EBRL_OK;
}

}  // extern "C"
