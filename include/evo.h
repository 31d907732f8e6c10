/*
 * evo.h -- C ABI of the schedule-driven cached denoising loop (EVO,
 * arXiv 2607.20293) on AMD Instinct MI355X (gfx950).
 *
 * The method (Sec. 3.1, Eq. 1): a pretrained transformer diffusion policy
 * runs T reverse denoising steps; the self-attention, cross-attention and
 * feed-forward residual branches of its L decoder layers are B = 3L
 * cacheable units.  A schedule S, a subset of the unit x step lattice with
 * |S| = K (Eq. 2, Eq. 3), decides where a unit's residual branch is
 * evaluated (and its cache refreshed); everywhere else the unit adds the
 * residual cached at its most recent refresh.  Caches are reset at the
 * start of every action query (Sec. 3.1, Sec. 3.4).  Weights, sampler and
 * action interface are those of the unchanged policy.
 *
 * Conventions for every call:
 *  - Return value: EVO_OK (0) or a negative EVO_E_* code; evo_last_error()
 *    then returns a thread-local message.  Every argument is validated
 *    before any device work is enqueued; on error nothing is enqueued and
 *    the policy is unchanged.
 *  - "host" pointers are ordinary CPU memory, read during the call only
 *    (copied; the caller may free them on return).  "device" pointers are
 *    HIP device memory on the policy's device; they stay owned by the
 *    caller and must stay valid until the enqueued work completes.
 *  - A policy is bound to the HIP device that was current at creation.
 *    Calls on one policy are not thread-safe.
 */
#ifndef EVO_H
#define EVO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  EVO_OK = 0,
  EVO_E_INVALID = -1,     /* bad argument (shape, value, NULL pointer, id) */
  EVO_E_STATE = -2,       /* call not valid in the current state (e.g. unknown schedule) */
  EVO_E_NOMEM = -3,       /* device or pinned host allocation failed */
  EVO_E_HIP = -4,         /* HIP runtime error (message has the HIP error string) */
  EVO_E_UNSUPPORTED = -5  /* valid request outside the compiled shape set */
};

enum { EVO_FP32 = 0, EVO_BF16 = 1 };          /* matmul operand precision */
enum { EVO_GRAN_LAYER = 0, EVO_GRAN_UNIT = 1 };/* lattice rows = L layers or 3L units */
enum { EVO_COLD_COMPUTE = 0, EVO_COLD_ZERO = 1 };

/* Policy shape and options.
 *   n_layers L, d_model d, n_heads h (d % h == 0), d_ff, horizon H (action
 *   tokens), action_dim A, n_obs_tokens, obs_dim, n_steps T.
 *   dtype: EVO_BF16 multiplies the projection matrices (obs projection,
 *     QKV, attention outputs, cross-attention Q and KV, MLP) in bfloat16
 *     (weights rounded to nearest even at creation) with fp32 accumulation;
 *     EVO_FP32 keeps them fp32.  The residual stream, LayerNorm statistics,
 *     softmax, GELU, embeddings, head and sampler are fp32 in both modes.
 *   cold_policy: what a unit does at a step where it is not scheduled but
 *     has never been refreshed in this query.  Eq. 1 leaves it open (the
 *     caches are reset per query).  EVO_COLD_COMPUTE evaluates every unit at
 *     step 0 (S' = S u B x {0}); EVO_COLD_ZERO adds a zero residual.
 *   clip_sample: nonzero clips the sampler's x0 estimate to [-1, 1].
 *   max_batch: largest batch evo_denoise accepts (sizes the caches).
 *   max_schedules: number of schedule ids (0 .. max_schedules-1). */
typedef struct {
  int32_t n_layers, d_model, n_heads, d_ff, horizon, action_dim;
  int32_t n_obs_tokens, obs_dim, n_steps;
  int32_t dtype, cold_policy, clip_sample;
  int32_t max_batch, max_schedules;
} evo_policy_desc;

/* Bookkeeping of the last evo_denoise call, summed over the batch.
 * Refreshes count unit positions (b, t) of the effective schedule.  FLOPs
 * count 2 per multiply-add of the matrix products (attention score and
 * value products dense) following Tables 1-3's "FLOPs for action
 * generation":
 *   per sample and evaluation  F_SA  = 2(4 H d^2 + 2 H^2 d)
 *                              F_CA  = 2(2 H d^2 + 2 S d^2 + 2 H S d)
 *                              F_FFN = 4 H d d_ff          (S = 1 + n_obs)
 *   always-on per step 4 H A d, per query 2 n_obs obs_dim d.
 * flops_kernel is what this implementation multiplies: the cross-attention
 * key/value products of the observation tokens are done once per query and
 * those of the time token once per policy, so they are not repeated at
 * each refresh.  Policies of width 256 whose n_heads x S <= 16 run the
 * cross-attention folded: W_q and W_o2 are applied once per memory token
 * (per query for the observation tokens, at creation for the time token)
 * and an evaluation multiplies only against the S x n_heads folded
 * columns, so there F_CA counts 2(2 H S n_heads d) per evaluation and the
 * query adds 4 n_obs d^2 per layer for the fold.  The byte counters are this implementation's algorithmic
 * traffic: cache reads/writes of reused/refreshed residuals (fp16 values
 * with bf16 operands, fp32 with fp32 operands), and weight
 * bytes of evaluated units summed over workgroups.  n_tiles counts the
 * sample tiles, n_workgroups the workgroups launched (small batches run
 * several workgroups per one-sample tile; each keeps its own caches, so the
 * cache bytes scale with it, while a unit's weights are split among them). */
typedef struct {
  uint64_t refreshes_requested;
  uint64_t refreshes_effective;
  uint64_t flops_cacheable;
  uint64_t flops_always;
  uint64_t flops_full;
  uint64_t flops_kernel;
  uint64_t cache_bytes_read;
  uint64_t cache_bytes_written;
  uint64_t weight_bytes;
  uint64_t n_tiles;
  uint64_t n_workgroups;
} evo_stats;

typedef struct evo_policy evo_policy;

/* Number of floats of the flat weight vector for `desc`, or a negative
 * EVO_E_* code.  Host-only; no device needed.
 * Flat order (Linear layers [out][in]):
 *   W_in[d][A] b_in[d] P_act[H][d] W_obs[d][obs_dim] b_obs[d] P_mem[1+n_obs][d]
 *   per layer l: ln1_g[d] ln1_b[d] W_qkv[3d][d] b_qkv[3d] W_o[d][d] b_o[d]
 *                ln2_g ln2_b W_q[d][d] b_q[d] W_kv[2d][d] b_kv[2d] W_o2[d][d] b_o2[d]
 *                ln3_g ln3_b W_1[d_ff][d] b_1[d_ff] W_2[d][d_ff] b_2[d]
 *   lnf_g[d] lnf_b[d] W_out[A][d] b_out[A]
 * Model (pre-norm decoder layers, LayerNorm eps 1e-5, exact-erf GELU):
 *   memory tokens mem = [sinusoid(k); obs W_obs^T + b_obs] + P_mem, k = T-1-t
 *   h = x W_in^T + b_in + P_act
 *   SA  = W_o . causal multi-head attention(LN1(h))     (scale 1/sqrt(d/h))
 *   CA  = W_o2 . attention(LN2(h) W_q^T, mem W_kv^T)   (unmasked)
 *   FFN = W_2 . GELU(W_1 . LN3(h) + b_1) + b_2
 *   eps = LN_f(h) W_out^T + b_out; DDPM step with squared-cosine betas
 *   (s = 0.008, cap 0.999), fixed-small variance, k-th step adds noise
 *   unless k == 0. */
int64_t evo_weight_count(const evo_policy_desc* desc);

/* Validate a descriptor without creating anything (host-only).  Returns
 * EVO_OK, EVO_E_INVALID or EVO_E_UNSUPPORTED (shape not compiled). */
int evo_check_desc(const evo_policy_desc* desc);

/* Create a policy on the current HIP device.
 *   host_weights: host float[n_floats] in the order above, n_floats ==
 *   evo_weight_count(desc).  Copied and re-laid-out on the device; the call
 *   returns after the device copies are complete.
 *   out: receives the policy handle (unchanged on error). */
int evo_create_policy(const evo_policy_desc* desc, const float* host_weights,
                      size_t n_floats, evo_policy** out);

/* Register (or replace) schedule `schedule_id` (Eq. 2): host uint8
 * lattice[rows][n_steps], row-major, entries 0 or 1 (1 = evaluate the unit
 * and refresh its cache at that step).  rows == L with EVO_GRAN_LAYER (a row
 * applies to the SA, CA and FFN units of its layer; the three residuals are
 * then cached as one sum) or 3L with EVO_GRAN_UNIT (row 3l+u, u = 0 SA,
 * 1 CA, 2 FFN).  n_steps must equal T; row index t is the t-th reverse
 * step, t = 0 the first (noisiest).  Host-only state; takes effect for
 * later evo_denoise calls. */
int evo_set_schedule(evo_policy* p, int32_t schedule_id, const uint8_t* lattice,
                     int32_t rows, int32_t n_steps, int32_t granularity);

/* Eq. 3 form of evo_set_schedule: K unique (row, step) pairs, host
 * int32 pairs[K][2].  Duplicates or out-of-range pairs -> EVO_E_INVALID. */
int evo_set_schedule_pairs(evo_policy* p, int32_t schedule_id, const int32_t* pairs,
                           int32_t K, int32_t granularity);

/* One action query per sample: run T cached denoising steps for `batch`
 * independent samples and write the final chunk x_0.
 *   obs_cond:  device float[batch][n_obs][obs_dim]
 *   noise:     device float[T][batch][H][A]; slice 0 is x_T, slice t+1 the
 *              standard-normal noise added after step t
 *   schedule_ids: host int32[batch] (NULL = all 0); each id must be
 *              registered.  Samples may carry different schedules.
 *   actions_out: device float[batch][H][A]
 *   hip_stream: hipStream_t to enqueue on (NULL = default stream).
 * Caches are reset for every call.  Asynchronous: returns after enqueueing;
 * the statistics of the call are available immediately (host computed). */
int evo_denoise(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                const int32_t* schedule_ids, float* actions_out, void* hip_stream);

/* For callers that cannot allocate memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation.  The same
 * computation and arguments as evo_denoise, and the same plan, kernels and
 * results; the kernels' working data (per-tile residual caches,
 * observation keys/values or fold records, the small-batch team exchange
 * slots, counters and error flag, and the call's plan) live in a fixed
 * device array of evo_noalloc_scratch_bytes() bytes (64 MiB) instead of the
 * policy's buffers.  The library looks up each device's copy of that array
 * once, when the first policy is created on the device; the array is held
 * until the process ends.  The call allocates nothing (no device, pinned or
 * host heap memory): the plan is built in arrays sized at evo_create_policy
 * and staged through the policy's pinned buffers.  A batch whose working
 * data does not fit the array is refused with EVO_E_UNSUPPORTED before
 * anything is enqueued (Push-T-shaped policies: about 200 samples with bf16
 * operands, about 120 with fp32).  Every
 * call on a device shares that device's array, which keeps the last call's
 * contents (each call clears what must start at zero): calls that overlap
 * on one device race (different policies, or different threads); calls of
 * one policy on different streams are ordered as for evo_denoise.
 * Enqueued on a stream that is being captured into a HIP graph, the call is
 * recorded (kernels, a fill kernel for the counters, and the copy of the
 * plan from the policy's pinned staging buffer); each replay reads the plan
 * that buffer holds when it runs, so replays stay valid while the policy's
 * calls after the capture use the same batch and schedule ids (they stage
 * the same bytes), and a replay is a call on the device's array like any
 * other.  evo_debug_read_cache refers to evo_denoise calls only
 * (EVO_E_STATE after this call). */
int evo_denoise_noalloc(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                        const int32_t* schedule_ids, float* actions_out, void* hip_stream);

/* Size in bytes of the per-device scratch array of evo_denoise_noalloc. */
size_t evo_noalloc_scratch_bytes(void);

/* Wait for the policy's last evo_denoise and report a device-side failure.
 * Small batches run a variant in which several workgroups share a tile and
 * meet at bounded device-side barriers; if one of those waits ever times
 * out, the kernel stops early, its outputs are invalid, and this call
 * returns EVO_E_HIP (the flag is then cleared; until it is, later team
 * launches stop at their first barrier).  Environment variables read by
 * evo_create_policy: EVO_TEAM=0 disables that variant, EVO_TEAM=<n> keeps
 * only teams of n workgroups (of those compiled); EVO_TEAM_SPIN_LIMIT
 * sets the number of polls before a wait gives up (default 2^20, about a
 * second; checked every 32 polls, so smaller values act as 32).  The test
 * hook evo_debug_team_withhold forces this error path from the host. */
int evo_synchronize(evo_policy* p);

/* ---- Redundancy-aware initialisation of the schedule search (Sec. 3.3,
 * Eq. 6 and Eq. 7).  Offline tooling around the cached loop: activations of
 * the uncached policy, their cross-step cosine dissimilarity, and the guided
 * sampling distribution over block x step positions. */

/* evo_denoise that also records, for every sample n, unit b (3L units,
 * row 3l+u, u = 0 SA, 1 CA, 2 FFN) and step t that is evaluated, the unit's
 * residual a_{n,b,t} (the branch output after its bias, before the residual
 * add) into acts_out: device float [batch][3L][T][H][d], caller-owned,
 * 3L*T*H*d floats per sample.  Positions that are not evaluated are left
 * untouched, so Sec. 3.3's activations of the uncached policy come from an
 * all-refresh schedule.  Each sample is one query r of Eq. 6.  Other
 * arguments, errors and asynchrony as evo_denoise. */
int evo_collect_activations(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                            const int32_t* schedule_ids, float* actions_out, float* acts_out, void* hip_stream);

/* Eq. 6: scores_out[b][t] = mean over the queries r < rollouts of
 * 1/(T-1) sum_{t' != t} (1 - cos(a_{r,b,t}, a_{r,b,t'})), the cosine of a
 * zero vector taken as 0.  acts: device float [rollouts][3L][T][H][d] as
 * written by evo_collect_activations; scores_out: device float [3L][T].
 * Computed in fp32 (step x step Gram matrices on fp32 MFMA, queries averaged
 * in order, deterministic).  rollouts in [1, max_batch]; 2 <= T <= 128 else
 * EVO_E_UNSUPPORTED.  Asynchronous on hip_stream; uses a per-policy
 * workspace, so calls on one policy must not overlap. */
int evo_redundancy_scores(evo_policy* p, int32_t rollouts, const float* acts, float* scores_out,
                          void* hip_stream);

/* Eq. 7 on the host: the scores (host float [rows][n_steps]) are normalised
 * to w in [0, 1] by min-max over all positions (all zeros if constant), and
 * probs_out[i] = (eps + w_i)^gamma / sum_j (eps + w_j)^gamma (host double,
 * same shape).  eps, gamma >= 0; the paper gives no values for them. */
int evo_guided_probabilities(const float* scores, int32_t rows, int32_t n_steps, double eps, double gamma,
                             double* probs_out);

/* K distinct positions drawn one after another without replacement from
 * probs (host double [rows][n_steps]), as for an initial individual of the
 * search (Sec. 3.3).  Implemented as the K largest keys log p - log(-log u)
 * (Gumbel-top-K, which has exactly that law) with the caller's uniforms
 * (host double [rows][n_steps], each in (0, 1)); equal keys go to the lower
 * flat index.  pairs_out: host int32 [K][2] = (row, step), in flat order;
 * feed it to evo_set_schedule_pairs.  K larger than the number of positions
 * with p > 0 -> EVO_E_INVALID. */
int evo_guided_sample(const double* probs, int32_t rows, int32_t n_steps, int32_t K, const double* uniforms,
                      int32_t* pairs_out);

/* ---- Schedule search (Sec. 3.2 with Eq. 4 and Eq. 5; Sec. 3.3 with Eq. 7,
 * Eq. 8 and Eq. 9; population settings of Sec. 4.1).  Offline: finds a
 * fixed-budget schedule for the cached loop by evolutionary search.
 *
 * A schedule (individual) is K distinct flat positions p = b*T + t of the
 * rows x T lattice (rows = 3L units or L layers), sorted ascending; that
 * array is its signature.  Randomness: Philox4x64-10 (Salmon et al., SC
 * 2011), key (seed, 0), counter (generation, purpose << 32 | slot, index, 0),
 * first output word w; uniform (0, 1) = ((w >> 12) + 1/2) 2^-52, integer
 * [0, n) = ((w >> 32) n) >> 32.  Purposes: 1 initial individual, 2
 * tournament, 3 crossover, 4 mutation test, 5 mutation target, 6 repair
 * drop, 7 repair fill; slot = individual or child index; index = a lattice
 * position (guided draws), a rank, an entrant or a draw number.
 *
 * Operators (the paper names them without parameters; these are the
 * readings):
 *  - initial population: individuals 0 .. n_guided-1 take K positions from
 *    Eq. 7's probabilities (evo_guided_sample with the purpose-1 uniforms of
 *    every position), the others are uniform K-subsets built by `fill`
 *    (below) from the empty set;
 *  - fill: draw j = 0, 1, ... adds position [0, N) of word j unless present,
 *    until K (after 64 N draws the missing positions are added in ascending
 *    order; never reached in practice);
 *  - ranking: fitness descending, ties to the lower population index; the
 *    next population is the n_elite best in that order, then the children;
 *  - tournament: `tournament` entrants drawn with replacement, highest
 *    fitness wins, ties to the lower index; two tournaments per child;
 *  - set-level crossover: positions of both parents kept; the r-th position
 *    (ascending) of those in one parent only is kept on bit r % 64 of word
 *    r / 64;
 *  - mutation: the r-th position (ascending) is replaced by a uniform
 *    lattice position (purpose 5, index r) when the 32-bit half r % 2 of
 *    word r / 2 is below floor(mutation_rate 2^32);
 *  - repair: duplicates merge; a surplus loses, one at a time, the element at
 *    index [0, size) of draw j = 0, 1, ... of the ascending list; a shortfall
 *    is completed by `fill` (purpose 7). */
typedef struct {
  int32_t K;                /* refreshes per schedule, 1 <= K <= rows*T (Eq. 5) */
  int32_t pop_size;         /* population size (Sec. 4.1: 30) */
  int32_t n_elite;          /* elites carried over, 0 .. pop_size (Sec. 4.1: 10) */
  int32_t max_generations;  /* evaluated populations, the initial one included (Sec. 4.1: 30) */
  int32_t tournament;       /* entrants per tournament, >= 1 */
  int32_t n_guided;         /* initial individuals drawn from Eq. 7, 0 .. pop_size */
  double mutation_rate;     /* in [0, 1] */
  uint64_t seed;            /* generator key */
} evo_ga_config;

typedef struct {
  int32_t generations;         /* populations evaluated */
  int32_t evaluations;         /* distinct schedules given a quick evaluation */
  int32_t memo_hits;           /* population members whose signature was already evaluated */
  int32_t formal_evaluations;  /* schedules given a formal evaluation (Eq. 8 trigger) */
  int32_t accepted;            /* 1: a schedule passed Eq. 9 and ended the search */
  int32_t reserved;
  double best_quick;           /* quick fitness of the returned schedule */
  double best_formal;          /* its formal score, NaN if it had none */
} evo_search_result;

/* Quick fitness of n schedules (host int32 [n][K]) into fitness_out (host
 * double [n]); formal score of one schedule (host int32 [K]).  Return 0, or
 * nonzero to abort the search (EVO_E_STATE). */
typedef int (*evo_quick_fn)(void* user, int32_t n, const int32_t* schedules, double* fitness_out);
typedef int (*evo_formal_fn)(void* user, const int32_t* schedule, double* score_out);

/* The initial population (host int32 [pop_size][K]).  probs: Eq. 7
 * probabilities, host double [rows][n_steps], needed when n_guided > 0
 * (else may be NULL); K must not exceed the positions with p > 0. */
int evo_ga_initial_population(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, const double* probs,
                              int32_t* pop_out);

/* Population `generation` (>= 1) from population generation-1 (host int32
 * [pop_size][K], each sorted and duplicate-free) and its fitness (host
 * double [pop_size], no NaN): elites, then children by tournament,
 * crossover, mutation and repair. */
int evo_ga_next_generation(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, int32_t generation,
                           const int32_t* pop, const double* fitness, int32_t* next_out);

/* The search loop on the host with caller-supplied fitness.  Each
 * generation, the schedules whose signature has no fitness yet are passed to
 * `quick` once (in population order, duplicates once); results are
 * memoised.  Early stopping (formal != NULL): after a generation is
 * evaluated, its members with quick fitness >= q_base (Eq. 8) that were not
 * formally evaluated before get `formal`, best first; the first with score
 * >= q_base - delta_acc (Eq. 9) is returned with accepted = 1.  Otherwise
 * the best member of the last population is returned.  best_out: host int32
 * [K].  pop_history (host int32 [max_generations][pop_size][K]) and
 * fit_history (host double [max_generations][pop_size]) may be NULL; the
 * first `generations` entries are written. */
int evo_ga_search(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, const double* probs,
                  evo_quick_fn quick, evo_formal_fn formal, void* user, double q_base, double delta_acc,
                  evo_search_result* result, int32_t* best_out, int32_t* pop_history, double* fit_history);

/* Fitness on the GPU for evo_search: a synthetic stand-in for Eq. 4's
 * rollout success rate (no simulator): episode n of a schedule succeeds when
 * its action chunk stays within tau (max-abs over H x A, decided in fp32) of
 * the chunk of the uncached policy (every unit evaluated at every step) for
 * the same observation and noise; the fitness is the fraction of successes.
 * The uncached policy scores 1, so q_base = 1 is Eq. 8's target. */
typedef struct {
  int32_t granularity;  /* EVO_GRAN_UNIT (rows 3L) or EVO_GRAN_LAYER (rows L) */
  int32_t n_quick;      /* quick episodes, >= 1; pop_size * n_quick <= max_batch */
  int32_t n_formal;     /* formal episodes (independent seeds), 0 = no early stopping; <= max_batch */
  float tau;            /* success threshold, >= 0 */
  double q_base;        /* Eq. 8 target */
  double delta_acc;     /* Eq. 9 allowed drop, >= 0 */
} evo_search_options;

/* The search with GPU fitness: every generation's new schedules are
 * evaluated in one evo_denoise call (schedule j on episodes j*n_quick ..
 * (j+1)*n_quick-1, the same n_quick observations and noises for every
 * schedule), deviations from the uncached chunks reduced on the device.
 * obs_quick, noise_quick: device, [n_quick][n_obs][obs_dim] and
 * [T][n_quick][H][A] as for evo_denoise; obs_formal, noise_formal the same
 * for n_formal episodes (NULL if n_formal == 0).  probs, result, best_out,
 * histories as evo_ga_search.  Needs pop_size <= max_schedules; the search
 * overwrites schedule ids 0 .. pop_size-1 (their contents afterwards are
 * unspecified).  Allocates and frees its own device workspace; synchronous
 * (returns when the search is done); runs on hip_stream.  Every denoising
 * call of the search runs one workgroup per sample tile, whatever its
 * batch (no small-batch teams): those variants give a sample the same bits
 * at any batch size, so a schedule's fitness does not depend on how many
 * schedules its generation evaluates.  A policy created with EVO_TEAM=0
 * reproduces a search's chunks bit for bit through evo_denoise. */
int evo_search(evo_policy* p, const evo_ga_config* cfg, const evo_search_options* opt, const float* obs_quick,
               const float* noise_quick, const float* obs_formal, const float* noise_formal, const double* probs,
               evo_search_result* result, int32_t* best_out, int32_t* pop_history, double* fit_history,
               void* hip_stream);

/* Statistics of the last evo_denoise call (host struct). */
int evo_get_stats(const evo_policy* p, evo_stats* out);

/* Measurement of the denoising kernel alone (Sec. 4.1 reports the cost of
 * the cached loop; this isolates its kernel from the per-query observation
 * pre-pass launched before it on the same stream).  With enable != 0, every
 * later evo_denoise records a pair of timing events on its stream around the
 * denoising kernel's launch (a ring of 64 pairs created here; a pair still
 * in use is waited for and harvested before it is recorded again).
 * enable == 0 stops the recording and destroys the events.  Errors:
 * EVO_E_INVALID for a NULL policy, EVO_E_HIP if an event cannot be created
 * (timing then stays off). */
int evo_set_kernel_timing(evo_policy* p, int32_t enable);

/* Waits for every recorded pair, then returns in *ms_total the summed
 * duration (milliseconds) and in *launches the number of denoising-kernel
 * launches timed since the last call of this function, and restarts both
 * sums at zero.  ms_total and launches are host pointers (either may be
 * NULL).  Errors: EVO_E_INVALID for a NULL policy, EVO_E_HIP from an event
 * query. */
int evo_kernel_time(evo_policy* p, double* ms_total, int64_t* launches);

/* Host-only bookkeeping for lattices without a policy: n_lat lattices
 * (host uint8[n_lat][rows][T]) of one granularity, per-sample ids (host
 * int32[batch]).  Fills refreshes and the FLOP fields of `out` as
 * evo_denoise would; byte and tile fields are zero. */
int evo_schedule_stats(const evo_policy_desc* desc, const uint8_t* lattices, int32_t n_lat,
                       int32_t rows, int32_t granularity, const int32_t* ids, int32_t batch,
                       evo_stats* out);

/* Host-only: per-(unit, step) execution codes of one lattice, host
 * uint8 out[3L][T].  Bit 0: evaluate; bit 1: store the cache after it;
 * bit 2: add the cached residual; bit 3: layer-merged cache.  For tests. */
int evo_schedule_codes(const evo_policy_desc* desc, const uint8_t* lattice, int32_t rows,
                       int32_t granularity, uint8_t* out);

/* Test hook: enable != 0 makes team member 0 of later evo_denoise calls
 * withhold its partial residuals, so that the other members' bounded waits
 * time out and the error path of evo_synchronize can be exercised (the
 * outputs of those calls are invalid); 0 restores normal calls.  Errors:
 * EVO_E_INVALID for a NULL policy. */
int evo_debug_team_withhold(evo_policy* p, int32_t enable);

/* Test hook: synchronise the policy's device and copy the cached residual
 * of `unit` for `sample` of the last evo_denoise into host float[H][d]
 * (for a layer-granular schedule, unit 3l+2 holds the layer's merged sum;
 * with bf16 operands the caches hold fp16 values, clamped to +-65504). */
int evo_debug_read_cache(evo_policy* p, int32_t unit, int32_t sample, float* host_dst);

/* Release all device and host resources (NULL is a no-op).  Synchronises
 * the policy's device first. */
void evo_destroy_policy(evo_policy* p);

/* ---- Observation encoder --------------------------------------------
 * The image policies turn camera frames into observation features with a
 * pretrained encoder that the method leaves unchanged (Sec. 3.1, Sec. 3.4;
 * the appendix's wall-clock table times action generation with visual
 * encoding included).  The paper prints no architecture; this library
 * builds a ResNet-18-topology network with GroupNorm in place of
 * BatchNorm and global average pooling, no final linear layer:
 *   stem: conv 7x7 stride 2 (pad 3), GroupNorm, ReLU, max pool 3x3 stride 2
 *   (pad 1); stage s (0-based), block b: y = ReLU(GN(conv3x3(ReLU(GN(
 *   conv3x3_stride(x))))) + sc(x)), stride 2 for b == 0 and s > 0,
 *   sc = GN(conv1x1_stride(x)) where the stride or width changes, else x;
 *   features = mean over the final map's pixels.
 * Convolutions have no bias; GroupNorm: groups of gn_group consecutive
 * channels, population variance over the group's channels and pixels,
 * eps 1e-5, per-channel gain and shift. */
typedef struct {
  int32_t height, width; /* image size, 8 .. 4096 */
  int32_t in_ch;         /* image channels, 1 .. 64 */
  int32_t stem_ch;       /* stem width, a multiple of 8 and of gn_group
                            (not a multiple of 8: EVO_E_UNSUPPORTED) */
  int32_t n_stages;      /* 1 .. 4 */
  int32_t widths[4];     /* stage widths, multiples of 8 and of gn_group, <= 4096 */
  int32_t blocks[4];     /* basic blocks per stage, 1 .. 16 */
  int32_t gn_group;      /* channels per GroupNorm group: 4, 8, 16, 32 or 64
                            (others: EVO_E_UNSUPPORTED) */
  int32_t dtype;         /* EVO_BF16: convolution operands rounded to bf16
                            (fp32 accumulation); EVO_FP32: fp32 operands */
  int32_t max_batch;     /* largest batch of evo_encode, 1 .. 65536; also
                            max_batch * height * width < 2^31 and the largest
                            activation map of max_batch images < 2^31 floats
                            (EVO_E_UNSUPPORTED otherwise) */
} evo_encoder_desc;

typedef struct evo_encoder evo_encoder;

/* Number of floats of the encoder's flat parameter array, or a negative
 * EVO_E_* code.  Order: "stem" conv [stem_ch][7][7][in_ch], its GroupNorm
 * gain [stem_ch] and shift [stem_ch]; then per stage and block: conv a
 * [c][3][3][cin], gain, shift; conv b [c][3][3][c], gain, shift; and where
 * the shortcut is projected, conv d [c][1][1][cin], gain, shift.  Host-only. */
int64_t evo_encoder_weight_count(const evo_encoder_desc* desc);

/* Build an encoder on the current HIP device.  host_weights: host float
 * [n_floats] in the order above (copied; the caller keeps ownership).
 * Allocates the packed weights and activation buffers for max_batch images.
 * Errors: EVO_E_INVALID (desc, n_floats, image too small for the network),
 * EVO_E_UNSUPPORTED, EVO_E_NOMEM, EVO_E_HIP.  On error *out is untouched. */
int evo_create_encoder(const evo_encoder_desc* desc, const float* host_weights, size_t n_floats,
                       evo_encoder** out);

/* Encode `batch` images.  images: device float [batch][height][width]
 * [in_ch] (NHWC), read only, 16-byte aligned (EVO_E_INVALID otherwise).  features_out: device float, row n at
 * features_out + n * out_stride holds widths[n_stages-1] features (so
 * features can be written straight into a policy's observation rows);
 * other elements are not touched.  Asynchronous on hip_stream (NULL = the
 * null stream); uses the encoder's activation buffers, so calls on one
 * encoder must not overlap.  The work split (convolution K splits,
 * GroupNorm statistics chunks) is planned for max_batch, so an image's
 * features are bitwise the same at every batch size of one encoder and do
 * not depend on the other images; encoders created with different
 * max_batch may differ in the last bits.  A batch well below max_batch runs
 * that plan on fewer workgroups. */
int evo_encode(evo_encoder* e, int32_t batch, const float* images, float* features_out, int32_t out_stride,
               void* hip_stream);

/* Convolution FLOPs of one evo_encode of `batch` images (2 per
 * multiply-add; normalisation and pooling not counted).  Host-only. */
int evo_encoder_flops(const evo_encoder* e, int32_t batch, uint64_t* flops_out);

/* Release the encoder (NULL is a no-op); synchronises its device first. */
void evo_destroy_encoder(evo_encoder* e);

/* Thread-local message of the last failed call on this thread. */
const char* evo_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* EVO_H */
