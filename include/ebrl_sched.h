/*
 * ebrl_sched.h -- the rollout-side scheduler that feeds the generation
 * calls: environment groups pipelined between simulation and generation
 * (Section 4.2.2, intra-rollout simulation-generation pipeline) and
 * step-level greedy core rebinding (Section 4.2.3 and Algorithm 2, with the
 * ready set of Eq. (1)).  Host code only: no call here touches a GPU.
 *
 * Model.  n_envs environments are split into n_groups contiguous groups
 * (group g holds envs [g * n_envs / n_groups, (g + 1) * n_envs / n_groups)).
 * Generation hands a whole group its next action chunk of chunk_len actions
 * at once (ebrl_sched_deliver); each env then steps through its chunk on
 * whatever CPU core frees up, independently of the others.  When every env
 * of a group has finished its chunk, the group's observations join the
 * generation queue (FIFO); the generation stage pops groups from it
 * (ebrl_sched_next_group) and runs them as one ragged batch.  At creation no
 * env holds actions and every group is queued, in group order.
 *
 * Algorithm 2 on a free core (ebrl_sched_dispatch): the ready set is the
 * envs with unfinished actions in their current chunk, no step in flight,
 * and a chunk delivered (Eq. (1)); the env with the longest recorded step
 * duration is chosen and marked running in the same locked operation, envs
 * with no recorded step first, ties by the lowest env id.  The caller binds
 * that env's worker to the core and runs one step; ebrl_sched_complete
 * records the step's duration, advances the env's action index and clears
 * its running mark.
 *
 * Readings of what the paper leaves open: a group enters generation only
 * when all its envs have finished their chunk (no partial groups); the
 * generation queue is served in the order groups completed; the bounded
 * queue's capacity does not change the order, so it is not modelled.
 *
 * Threading: every call takes the scheduler's lock, so several core threads
 * and the generation thread may call concurrently.  Status codes are those
 * of ebrl.h.
 */
#ifndef EBRL_SCHED_H
#define EBRL_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ebrl_sched ebrl_sched;

/* EBRL_E_INVALID unless 1 <= n_groups <= n_envs and chunk_len >= 1. */
int ebrl_sched_create(int32_t n_envs, int32_t n_groups, int32_t chunk_len, ebrl_sched** out);
void ebrl_sched_destroy(ebrl_sched* s);

/* Algorithm 2 for free core `core`: *env = the chosen env (now running), or
 * -1 if no env is ready (the core stays idle).  bind_stride 0 lets the core
 * take any ready env (the rebinding of Algorithm 2); bind_stride C > 0
 * restricts core c to envs with e % C == c, the fixed core assignment the
 * paper contrasts rebinding with (0 <= core < C required). */
int ebrl_sched_dispatch(ebrl_sched* s, int32_t core, int32_t bind_stride, int32_t* env);

/* The running step of `env` finished after `duration` seconds (>= 0).  If it
 * was the last unfinished action of its group's chunk, *group_done = 1 and
 * the group joins the generation queue; else 0.  EBRL_E_STATE if env has no
 * step in flight. */
int ebrl_sched_complete(ebrl_sched* s, int32_t env, double duration, int32_t* group_done);

/* Pops the oldest queued group: *group (or -1 if the queue is empty), its
 * env ids in env_ids[0 .. *n) (capacity `cap`, EBRL_E_INVALID if too small). */
int ebrl_sched_next_group(ebrl_sched* s, int32_t* group, int32_t* env_ids, int32_t cap, int32_t* n);

/* Generation produced `group`'s next chunk: each of its envs restarts at
 * action 0.  EBRL_E_STATE unless the group was popped and not yet
 * delivered. */
int ebrl_sched_deliver(ebrl_sched* s, int32_t group);

/* One env's state: actions done in the current chunk, whether a step is in
 * flight, whether a chunk is delivered, and its recorded step duration (a
 * negative value: none yet). */
int ebrl_sched_env_state(const ebrl_sched* s, int32_t env, int32_t* steps_done, int32_t* running,
                         int32_t* has_chunk, double* last_duration);

#ifdef __cplusplus
}
#endif
#endif /* EBRL_SCHED_H */
