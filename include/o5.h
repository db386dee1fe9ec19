/*
 * o5.h -- C ABI of libo5: one PPO optimizer step on a single-layer LSTM
 * policy, after "Dota 2 with Large Scale Deep Reinforcement Learning"
 * (OpenAI Five, arXiv:1912.06680), on AMD Instinct MI355X (gfx950).
 *
 * The paper's optimizer trains a central single-layer 4096-unit LSTM whose
 * state feeds linear policy and value heads, with PPO and generalized
 * advantage estimation, Adam, truncated backpropagation through time over
 * 16-timestep samples, and a per-parameter gradient clip to +-5 sqrt(v)
 * (section "Training System", subsections "Playing Dota using AI" and
 * "Optimizing the Policy"; Table "Hyperparameters").  Each call below is one
 * step of that computation.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument is a DEVICE pointer unless marked "host".  All
 *   device buffers belong to the caller; the library never allocates device
 *   memory, never keeps a pointer after it returns and never synchronises
 *   the stream.  Scratch space is passed in as (ws, ws_bytes); the matching
 *   *_workspace_bytes() query gives the size needed.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Work is enqueued in order on that stream; calls on different streams
 *   with disjoint buffers are independent.
 * - Arguments are validated on the host before anything is enqueued.  On
 *   error the call returns a nonzero O5_E_* code, enqueues nothing, leaves
 *   every output untouched and records a message for o5_last_error() (per
 *   calling thread).  Faults raised by the device while running enqueued
 *   work surface at the caller's next synchronisation, as for any HIP call.
 * - Device pointers must be 16-byte aligned.  Outputs are overwritten, never
 *   accumulated into; inputs and outputs must not overlap except where a
 *   call says so (o5_adam_step updates p, m, v in place).
 * - Results are deterministic: identical inputs on the same GPU give
 *   bitwise identical outputs (no floating-point atomics).
 * - Layouts are row-major and time-major: [T, B, D] means element
 *   (t, b, d) at index (t * B + b) * D + d.  LSTM gate blocks are ordered
 *   (i, f, g, o): row g * H + j of a [4H, .] weight holds gate g of unit j.
 * - bf16 buffers hold IEEE bfloat16 bit patterns (uint16).
 */
#ifndef O5_H
#define O5_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define O5_VERSION 100 /* 1.0.0 */

enum {
  O5_OK = 0,
  O5_E_NULL = 1,      /* a required pointer is NULL */
  O5_E_SHAPE = 2,     /* a size is out of range or inconsistent */
  O5_E_DTYPE = 3,     /* unknown o5_dtype */
  O5_E_ALIGN = 4,     /* a device pointer is not 16-byte aligned */
  O5_E_WORKSPACE = 5, /* ws is NULL or ws_bytes is below the query */
  O5_E_HIP = 6,       /* the HIP runtime refused a launch */
  O5_E_ARG = 7        /* another argument is out of range */
};

/* Arithmetic type of the GEMM inputs (x, weights, hidden state).  Cell
 * state, gradients, optimizer state, advantages and losses are always fp32;
 * GEMMs always accumulate in fp32.  Any other non-negative value is
 * rejected with O5_E_DTYPE (the last enumerator only widens the type's
 * range to every such value, so that a C caller's bad value is defined
 * behaviour on the C++ side as well). */
typedef enum { O5_F32 = 0, O5_BF16 = 1, O5_DTYPE_MAX_ENUM = 0x7fffffff } o5_dtype;

/* O5_VERSION of the loaded library. */
int o5_version(void);
/* Static description of a status code (never NULL). */
const char* o5_status_str(int status);
/* Message of the calling thread's last failed call ("" if none). */
const char* o5_last_error(void);

/* ------------------------------------------------------------------------
 * o5_lstm_fwd -- T steps of the single-layer LSTM over a minibatch of B
 * samples, each started from its stored rollout state (section "Training
 * System": a single-layer 4096-unit LSTM of the forget-gate kind (Gers et
 * al. 1999); subsection "Optimizing the Policy": samples of 16 timesteps).
 *
 *   h~ = (1 - reset[t,b]) h_{t-1},  c~ = (1 - reset[t,b]) c_{t-1}
 *   a  = W_x x_t + W_h h~ + b;  i, f, o = sigmoid(a_i, a_f, a_o);  g = tanh(a_g)
 *   c_t = f c~ + i g;  h_t = o tanh(c_t)            (h_{-1} = h0, c_{-1} = c0)
 *
 * dt       GEMM input type: x, Wx, Wh and the output h are fp32 (O5_F32) or
 *          bf16 (O5_BF16).
 * T, B     steps and samples, >= 1, B <= 2097088.  D, H: input width and
 *          hidden units, multiples of 64, <= 65536.  T*B*4H and T*B*D below
 *          2^31.
 * x        [T, B, D] dt.   Wx [4H, D] dt.   Wh [4H, H] dt.   b [4H] fp32.
 * h0, c0   [B, H] fp32, the start state of each sample.
 * reset    [T, B] uint8 or NULL (no resets): nonzero zeroes the carried
 *          state before step t of sample b.
 * h        out [T, B, H] dt.   c: out [T, B, H] fp32.
 * gates    out [T, B, 4H] dt, the post-activation (i, f, g, o) that
 *          o5_lstm_bptt needs; NULL for inference (nothing saved).
 * ws       scratch of o5_lstm_fwd_workspace_bytes(dt, T, B, D, H) bytes.
 * ------------------------------------------------------------------------ */
size_t o5_lstm_fwd_workspace_bytes(o5_dtype dt, int T, int B, int D, int H);
int o5_lstm_fwd(o5_dtype dt, int T, int B, int D, int H,
                const void* x, const void* Wx, const void* Wh, const float* b,
                const float* h0, const float* c0, const uint8_t* reset,
                void* h, float* c, void* gates,
                void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_lstm_bptt -- truncated backpropagation through time over the T steps
 * of one o5_lstm_fwd call (subsection "Optimizing the Policy": BPTT over
 * samples of 16 timesteps).  It differentiates
 *     J = sum_t <dh[t], h[t]> + <dhT, h[T-1]> + <dcT, c[T-1]>
 * with respect to the weights; no gradient flows into h0 or c0 (the
 * truncation).
 *
 * x, Wx, Wh, h0, c0, reset, h, c, gates: exactly as given to / produced by
 *          o5_lstm_fwd (gates must not be NULL).
 * dh       [T, B, H] fp32: gradient arriving at every step's output h[t]
 *          (from the heads).
 * dhT, dcT [B, H] fp32 or NULL (= 0): gradient arriving at the final state.
 * dWx      out [4H, D] fp32.   dWh: out [4H, H] fp32.   db: out [4H] fp32.
 * dx       out [T, B, D] dt, or NULL to skip the input gradient.
 * ws       scratch of o5_lstm_bptt_workspace_bytes(dt, T, B, D, H) bytes.
 * ------------------------------------------------------------------------ */
size_t o5_lstm_bptt_workspace_bytes(o5_dtype dt, int T, int B, int D, int H);
int o5_lstm_bptt(o5_dtype dt, int T, int B, int D, int H,
                 const void* x, const void* Wx, const void* Wh,
                 const float* h0, const float* c0, const uint8_t* reset,
                 const void* h, const float* c, const void* gates,
                 const float* dh, const float* dhT, const float* dcT,
                 float* dWx, float* dWh, float* db, void* dx,
                 void* ws, size_t ws_bytes, void* stream);

/* o5_lstm_bptt_factored -- o5_lstm_bptt (dt = O5_BF16 only) with the heads'
 * gradient given in factored form, dh[t] = P[t] W^T (P [T*B, ld] and W
 * [H, ld] bf16 as written by o5_ppo_loss_grad_factored over the N = T*B
 * rows; ld a multiple of 64, at most 4096): each step's recurrent product
 * takes [P_t | dG_{t+1}] against [W | W_h^T], so dh is never stored.  Same
 * workspace query as o5_lstm_bptt.  O5_E_DTYPE for fp32, O5_E_SHAPE for a
 * bad ld. */
int o5_lstm_bptt_factored(o5_dtype dt, int T, int B, int D, int H,
                          const void* x, const void* Wx, const void* Wh,
                          const float* h0, const float* c0,
                          const uint8_t* reset, const void* h, const float* c,
                          const void* gates, const uint16_t* P,
                          const uint16_t* W, int ld, const float* dhT,
                          const float* dcT, float* dWx, float* dWh, float* db,
                          void* dx, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_gae -- generalized advantage estimation over S rollout segments of L
 * steps (subsection "Optimizing the Policy": PPO with GAE, advantages
 * smoothed over 256-step segments; Table "Hyperparameters": lambda = 0.95).
 *
 *   delta_t = r_t + gamma (1 - done_t) v_{t+1} - v_t
 *   adv_t   = delta_t + gamma lambda (1 - done_t) adv_{t+1}    (adv_L = 0)
 *   ret_t   = adv_t + v_t
 *
 * L, S     >= 1.
 * r        [L, S] fp32 rewards.   v: [L+1, S] fp32 values, row L the
 *          bootstrap value after the segment.   done: [L, S] uint8, nonzero
 *          marks transition t terminal.
 * gamma, lambda in [0, 1].
 * adv, ret out [L, S] fp32.
 * ------------------------------------------------------------------------ */
int o5_gae(int L, int S, const float* r, const float* v, const uint8_t* done,
           float gamma, float lambda, float* adv, float* ret, void* stream);

/* ------------------------------------------------------------------------
 * o5_reward_process -- the reward post-processing ahead of GAE (appendix
 * "Reward Weights": zero sum, game time weighting, team spirit; Table
 * "Hyperparameters": rewards are normalised by a running estimate of their
 * standard deviation).  G games of two teams of five heroes; hero h of team
 * k in game g is segment s = 10 g + 5 k + h of the [L, S] layout that
 * o5_gae reads (S = 10 G).  For step t of game g and hero i of team A
 * (enemy team B):
 *
 *   rho_i = shaped_i * decay_base^(game_time / decay_minutes) + outcome_i
 *   z_i   = (1 - tau) rho_i + tau mean_{j in A} rho_j - mean_{j in B} rho_j
 *   r_i   = z_i / sqrt(var + eps)
 *
 * (team spirit mixes each hero's reward with its team's mean; the zero-sum
 * step subtracts the enemies' mean, which team spirit leaves unchanged).
 * var is the variance of every z seen so far: the running summary `stats`
 * = (count, mean, M2), M2 the sum of squared deviations from the mean, is
 * merged with this call's values (fp64, fixed order) and written back
 * before r is formed.  Start from stats = (0, 0, 0).
 *
 * L, G      >= 1, 10 L G < 2^31.
 * shaped    [L, S] fp32 raw shaped rewards.   outcome: [L, S] fp32 win/loss
 *           reward, not time-weighted, or NULL (= 0).   game_time: [L, G]
 *           fp32, minutes since the game began.
 * hp        tau in [0, 1] (0.3 in the paper's baseline); 0 < decay_base <= 1
 *           (0.6); decay_minutes > 0 (10); eps > 0 (1e-8).
 * stats     [3] fp64, updated in place.
 * r         out [L, S] fp32 (no overlap with the inputs).
 * ws        scratch of o5_reward_process_workspace_bytes(L, G) bytes.
 * ------------------------------------------------------------------------ */
typedef struct {
  float tau;           /* team spirit */
  float decay_base;    /* 0.6 */
  float decay_minutes; /* 10 */
  float eps;           /* 1e-8 */
} o5_reward_hp;

size_t o5_reward_process_workspace_bytes(int L, int G);
int o5_reward_process(int L, int G, const float* shaped, const float* outcome,
                      const float* game_time, o5_reward_hp hp, double* stats,
                      float* r, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_obs_normalize -- observation normalisation (appendix "Observation
 * Space": every float observation has a running mean and standard
 * deviation of all data ever observed subtracted and divided out, the
 * result clipped to (-5, 5)).  Per feature j the running summary (count,
 * mean, M2 = sum of squared deviations) is merged with this call's N rows
 * (fp64, fixed order) and written back; then
 *
 *   o[n, j] = clamp((obs[n, j] - mean_j) / sqrt(M2_j / count_j + eps), -clip, clip)
 *
 * dt       type of o (bf16: the operand of the pre-LSTM layer).
 * N >= 1 rows; Do features, a positive multiple of 4.
 * obs      [N, Do] fp32.   stats: [3, Do] fp64 (counts, means, M2),
 *          updated in place; start from zeros.
 * clip     5 in the paper; eps > 0 (1e-8) keeps a constant feature at 0.
 * o        out [N, Do] dt.   ws: o5_obs_normalize_workspace_bytes(N, Do).
 * ------------------------------------------------------------------------ */
size_t o5_obs_normalize_workspace_bytes(int N, int Do);
int o5_obs_normalize(o5_dtype dt, int N, int Do, const float* obs, double* stats,
                     float clip, float eps, void* o, void* ws, size_t ws_bytes,
                     void* stream);

/* ------------------------------------------------------------------------
 * o5_prelstm_fwd / o5_prelstm_bwd -- the layer between the flattened
 * observation and the LSTM (appendix "Neural Network Architecture": a
 * fully-connected layer, then a cross-hero pool that max-pools the first
 * 25% of the vector across the five replica networks of a team):
 *
 *   y = relu(o W^T + b)                                  [N, D] fp32
 *   x[n, j] = max over the 5 replicas of y[., j]  (j < D/4),  y[n, j] else
 *
 * The five replicas of a team are five consecutive samples b = 5 q + r of
 * the time-major [T, B, .] layout (B a multiple of 5), pooled at every
 * timestep.  The backward takes dx = dL/dx (from o5_lstm_bptt), sends the
 * pooled features' summed gradient to the first replica attaining the
 * maximum, applies the ReLU mask and returns
 *
 *   dW = dpre^T o  [D, Do] fp32,   db = sum_n dpre [D] fp32
 *
 * (bf16 path: dpre is rounded to bf16 as the operand of dW; db sums the
 * unrounded values).  No gradient reaches the observation.
 *
 * dt       type of o, W, x and dx.   T >= 1; B a positive multiple of 5 with
 *          T B / 5 <= 65535; Do and D positive multiples of 64.
 * o        [T B, Do] dt (from o5_obs_normalize).   W: [D, Do] dt.   b: [D].
 * y        out (fwd) / in (bwd) [T B, D] fp32: the layer's output before the
 *          pool, kept for the backward.   x: out [T B, D] dt, the LSTM input.
 * dx       [T B, D] dt.   dW, db: out.
 * ws       (bwd) o5_prelstm_bwd_workspace_bytes(dt, T, B, Do, D) bytes.
 * ------------------------------------------------------------------------ */
int o5_prelstm_fwd(o5_dtype dt, int T, int B, int Do, int D, const void* o,
                   const void* W, const float* b, float* y, void* x, void* stream);
size_t o5_prelstm_bwd_workspace_bytes(o5_dtype dt, int T, int B, int Do, int D);
int o5_prelstm_bwd(o5_dtype dt, int T, int B, int Do, int D, const void* o,
                   const float* y, const void* dx, float* dW, float* db,
                   void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_segments_to_samples -- cut each of S segments of L steps into L/T
 * samples of T steps, the unit truncated BPTT runs on (Figure "Timescales
 * and Staleness": a segment is subdivided into samples of 16 policy
 * actions).  Sample b = s * (L/T) + j holds segment steps T*j .. T*j+T-1.
 *
 * L, S, T  >= 1, T divides L.
 * adv, ret [L, S] fp32.   done: [L, S] uint8.
 * adv_s, ret_s out [T, B] fp32 (B = S*L/T).
 * reset    out [T, B] uint8: reset[0, b] = 0 and reset[t, b] = (done at the
 *          previous step of the same sample != 0) for t >= 1.
 * ------------------------------------------------------------------------ */
int o5_segments_to_samples(int L, int S, int T, const float* adv, const float* ret,
                           const uint8_t* done, float* adv_s, float* ret_s,
                           uint8_t* reset, void* stream);

/* ------------------------------------------------------------------------
 * o5_ppo_loss_grad -- policy and value heads, PPO loss and its gradient
 * (appendix "Neural Network Architecture": the action logits and the value
 * are linear projections of the LSTM state, sharing the network and its
 * gradients; appendix "Action Space": a factorised action with masking of
 * ignored parameter heads, each timestep's choice restricted by action
 * filters to the available actions; subsection "Optimizing the Policy" and Table
 * "Hyperparameters": PPO clipping 0.2, value loss weight 1.0; appendix
 * "Exploration", "Loss function": entropy bonus c S[pi], c = 0.01).
 *
 *   z = h Wp^T + bp;  head k = columns [o_k, o_k + n_k); value V = z[:, A]
 *   logpi = sum_k m_k log softmax(z_k)[a_k];  r = exp(logpi - logp_old)
 *   L = -mean min(r A, clip(r, 1-eps, 1+eps) A) + vf_coef mean (V - R)^2
 *       - ent_coef mean sum_k m_k S_k
 *
 * dt       type of h and Wp.   N: rows (timesteps), >= 1.   H: multiple of
 *          64.   K: heads, 1..8.   head_sizes: host [K], each >= 1, with
 *          A + 1 = sum + 1 <= 1024.
 * h        [N, H] dt.   Wp: [A+1, H] dt, last row the value head.   bp:
 *          [A+1] fp32.
 * act      [N, K] int32, action index within each head (0 <= a < n_k).
 * logp_old, adv, ret [N] fp32 (behaviour log-probability of the joint
 *          action, advantage, value target).
 * head_mask [N, K] uint8 or NULL (all heads count).
 * avail    [N, A] uint8 or NULL (all available): nonzero marks an available
 *          logit.  Each head's softmax runs over its available logits only;
 *          an unavailable logit gets probability 0 and no gradient; a head
 *          with no available logit in a row adds nothing; an unavailable
 *          taken action has log-probability -inf (ratio 0).  A head with
 *          head_mask 0 adds nothing in every case.
 * unit     host pointer to an o5_unit_head, or NULL.
 * hp       {clip_eps, vf_coef, ent_coef}.
 * stats    out [8] fp32: total, pg, vf, ent, clipfrac (mean |r-1| > eps),
 *          approx_kl (mean (r - 1) - log r), mean_ratio, nonfinite (rows
 *          whose loss term is not finite).
 * dh       out [N, H] fp32 = dL/dh.   dWp: out [A+1, H] fp32.   dbp: out
 *          [A+1] fp32.
 * ws       scratch of o5_ppo_loss_grad_workspace_bytes(...) bytes.
 * ------------------------------------------------------------------------ */
typedef struct {
  float clip_eps; /* 0.2 */
  float vf_coef;  /* 1.0 */
  float ent_coef; /* 0.01 */
} o5_ppo_hp;

/* Unit-selection head (appendix "Neural Network Architecture": the unit
 * embeddings of the observation processing travel beside the LSTM and the
 * action heads use them to choose a unit to target).  Head `head` scores its
 * n_head units against per-row embeddings instead of its rows of Wp, bp:
 *
 *   q = h Wq^T + bq [N, d],   z_head[n, u] = <q[n], E[n, u]>
 *
 * Those rows of Wp and bp are unused (o5_ppo_loss_grad writes zero gradient
 * for them); the gradient reaches Wq, bq and h through q, none goes to E.
 * Passed by host pointer; NULL = no such head. */
typedef struct {
  int head;        /* 0 <= head < K */
  int d;           /* query and embedding width, a power of two in 8..512 */
  const void* Wq;  /* [d, H] dt */
  const float* bq; /* [d] */
  const void* E;   /* [N, n_head, d] dt (rows as h) */
  float* dWq;      /* out [d, H] (o5_ppo_loss_grad only) */
  float* dbq;      /* out [d] (o5_ppo_loss_grad only) */
} o5_unit_head;

size_t o5_ppo_loss_grad_workspace_bytes(o5_dtype dt, int N, int H, int K,
                                        const int* head_sizes,
                                        const o5_unit_head* unit);
int o5_ppo_loss_grad(o5_dtype dt, int N, int H, int K, const int* head_sizes,
                     const void* h, const void* Wp, const float* bp,
                     const int32_t* act, const float* logp_old, const float* adv,
                     const float* ret, const uint8_t* head_mask,
                     const uint8_t* avail, const o5_unit_head* unit, o5_ppo_hp hp,
                     float* stats, float* dh, float* dWp, float* dbp,
                     void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * The heads' gradient in factored form (bf16 only; the same loss and
 * gradient as o5_ppo_loss_grad, appendix "Neural Network Architecture" and
 * subsection "Optimizing the Policy").  dL/dh is a product of a narrow
 * per-row gradient and the heads' weights, dh = P W^T, and the backward pass
 * can form it inside its own recurrent product instead of reading a
 * [N, H] fp32 dh:
 *
 *   P [N, ld] bf16: row n = [hi | lo], hi = bf16(g_n), lo = bf16(g_n - hi),
 *       g_n = (dL/dz_n, then dL/dq_n for a unit head), zero-padded to ld/2
 *   W [H, ld] bf16: row j = [w_j | w_j], w_j = (Wp[:, j], then Wq[:, j])
 *
 * o5_ppo_head_grad_ld returns ld for these heads (a multiple of 64; 0 if
 * they are invalid).  o5_ppo_loss_grad_factored takes the arguments of
 * o5_ppo_loss_grad, dt = O5_BF16, with P, W and ld in place of dh
 * (O5_E_DTYPE for fp32, O5_E_SHAPE if ld is not the value above); its
 * workspace query is o5_ppo_loss_grad_workspace_bytes.  stats, dWp, dbp and
 * the unit head's gradients are those of o5_ppo_loss_grad bit for bit.
 * ------------------------------------------------------------------------ */
int o5_ppo_head_grad_ld(int H, int K, const int* head_sizes,
                        const o5_unit_head* unit);
int o5_ppo_loss_grad_factored(o5_dtype dt, int N, int H, int K,
                              const int* head_sizes, const void* h,
                              const void* Wp, const float* bp,
                              const int32_t* act, const float* logp_old,
                              const float* adv, const float* ret,
                              const uint8_t* head_mask, const uint8_t* avail,
                              const o5_unit_head* unit, o5_ppo_hp hp,
                              float* stats, uint16_t* P, uint16_t* W, int ld,
                              float* dWp, float* dbp,
                              void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_adam_step -- Adam with the per-parameter clip of each gradient element
 * to +-clip_k sqrt(v) (subsection "Optimizing the Policy"; Table
 * "Hyperparameters": beta1 0.9, beta2 0.999, learning rate 5e-5):
 *
 *   v = b2 v + (1-b2) g^2;  vh = v / (1 - b2^step)
 *   g' = clamp(g, -clip_k sqrt(vh), clip_k sqrt(vh))     (clip_k <= 0: g' = g)
 *   m = b1 m + (1-b1) g';   mh = m / (1 - b1^step)
 *   p = p - lr mh / (sqrt(vh) + eps)
 *
 * n        elements (>= 1).   p, m, v: [n] fp32, updated in place.   g: [n]
 *          fp32.   p_bf16: out [n] bf16 copy of the new p, or NULL.
 * step     1-based step counter (>= 1).
 * ------------------------------------------------------------------------ */
typedef struct {
  float lr;     /* 5e-5 */
  float beta1;  /* 0.9 */
  float beta2;  /* 0.999 */
  float eps;    /* 1e-8 */
  float clip_k; /* 5; <= 0 turns the clip off */
} o5_adam_hp;

int o5_adam_step(size_t n, float* p, float* m, float* v, const float* g,
                 uint16_t* p_bf16, o5_adam_hp hp, int step, void* stream);

/* ------------------------------------------------------------------------
 * o5_policy_sample -- rollout inference heads: logits and value from the
 * LSTM state, then one action per head sampled from its categorical
 * distribution (section "Training System", subsection "Playing Dota using
 * AI": an action is sampled from the output distribution every timestep).
 * The draw is Gumbel-max, a = argmax_a (z_a + G_a), G = -ln(-ln U), with U
 * from Philox4x64-10 (Salmon et al., SC'11): the noise for logit a of head
 * k in row b is word (a mod 4) of the block with counter
 * (a div 4, k, b, counter) and key (seed, 0); U = ((word >> 40) + 0.5)/2^24.
 * Ties go to the lowest index.  Only available logits are drawn (appendix
 * "Action Space": action filters): the argmax and the log-sum-exp of the
 * log-probability run over them; the noise of a logit does not depend on
 * the mask.
 *
 * dt, B, H, K, head_sizes, h [B, H], Wp, bp: as for o5_ppo_loss_grad.
 * avail    [B, A] uint8 or NULL (all available), as for o5_ppo_loss_grad.
 * unit     host pointer to an o5_unit_head (dWq, dbq unused), or NULL.
 * act      out [B, K] int32; -1 for a head with no available logit.
 * logp     out [B] fp32, joint log-probability of the sampled action (heads
 *          with no available logit add nothing).   value: out [B] fp32.
 * ws       scratch of o5_policy_sample_workspace_bytes(...) bytes.
 * ------------------------------------------------------------------------ */
size_t o5_policy_sample_workspace_bytes(o5_dtype dt, int B, int H, int K,
                                        const int* head_sizes,
                                        const o5_unit_head* unit);
int o5_policy_sample(o5_dtype dt, int B, int H, int K, const int* head_sizes,
                     const void* h, const void* Wp, const float* bp,
                     const uint8_t* avail, const o5_unit_head* unit,
                     uint64_t seed, uint64_t counter,
                     int32_t* act, float* logp, float* value,
                     void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * o5_policy_sample_static -- o5_policy_sample without a workspace, for the
 * callers that cannot allocate: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Arguments, outputs and errors
 * are those of o5_policy_sample, and so are the results (the same kernels:
 * bitwise the same outputs).  It allocates nothing: its scratch is a device
 * array of O5_STATIC_SCRATCH_BYTES inside the library, one per GPU, held
 * until the process ends; its address on a GPU is looked up on the first
 * call there (with that GPU current) and kept.  A shape whose
 * o5_policy_sample_workspace_bytes exceeds O5_STATIC_SCRATCH_BYTES is
 * rejected with O5_E_SHAPE (with the paper's 75 logits at H = 4096 every
 * batch of up to 16,128 rows fits).  Every call on one GPU shares that GPU's array, which
 * keeps the last call's contents (no part of it needs to start at zero:
 * each call writes all it reads), so calls that overlap on one GPU -- two
 * streams, or two host threads -- race: serialise them.
 * ------------------------------------------------------------------------ */
#define O5_STATIC_SCRATCH_BYTES (16 << 20)
int o5_policy_sample_static(o5_dtype dt, int B, int H, int K, const int* head_sizes,
                            const void* h, const void* Wp, const float* bp,
                            const uint8_t* avail, const o5_unit_head* unit,
                            uint64_t seed, uint64_t counter,
                            int32_t* act, float* logp, float* value, void* stream);

/* ------------------------------------------------------------------------
 * Surgery on the flat parameter vector (appendix "Surgery"; subsection
 * "Continual Transfer via Surgery").  Layout of a vector for (D, H, A1):
 * Wx [4H, D], Wh [4H, H], b [4H], Wp [A1, H], bp [A1], fp32, gate blocks
 * (i, f, g, o) along 4H; o5_param_count(D, H, A1) gives its length (0 for
 * sizes < 1).  m and v are Adam's moments in the same layout.
 *
 * o5_surgery_widen -- widen the LSTM from H to H2 >= H units and extend its
 * input from D to D2 >= D features.  Old weights keep their places; the
 * LSTM's new weights (rows of new units, columns of Wh reading new units,
 * new biases) are scale * (2U - 1), U from Philox4x64-10 with counter
 * (e div 4, 0, 0, 0) and key (seed, 1), word e mod 4, for element e of the
 * new vector, U = ((word >> 40) + 1/2) / 2^24 (the paper used values much
 * smaller than the existing weights); columns of Wx reading new inputs and
 * columns of Wp reading new units are 0, so with scale = 0 the widened
 * network computes the old function exactly on the old units.  Old
 * parameters keep their moments, new ones start at 0 (the paper restarts
 * with learning rate 0 for a while: o5_adam_step with lr = 0 leaves p
 * bitwise unchanged while the moments adapt).
 * m_old, v_old may be NULL (zeros).  The new buffers must not overlap the
 * old ones.
 *
 * o5_surgery_fold_input -- the last D - Dk inputs of the LSTM are a constant
 * vector E [D - Dk] (appendix "Bloopers", subsection "Zero Team Spirit
 * Embedding": a constant input is a modified bias): b' = b + Wx[:, Dk:] E,
 * Wx' = Wx[:, :Dk], the rest copied; the dropped columns' moments are
 * discarded, every other parameter keeps its moments.  1 <= Dk < D.
 * ------------------------------------------------------------------------ */
size_t o5_param_count(int D, int H, int A1);
int o5_surgery_widen(int D, int H, int A1, int D2, int H2, const float* p_old,
                     const float* m_old, const float* v_old, float* p_new,
                     float* m_new, float* v_new, float scale, uint64_t seed,
                     void* stream);
int o5_surgery_fold_input(int D, int H, int A1, int Dk, const float* E,
                          const float* p_old, const float* m_old,
                          const float* v_old, float* p_new, float* m_new,
                          float* v_new, void* stream);

/* ------------------------------------------------------------------------
 * o5_f32_to_bf16 -- round n fp32 values to bfloat16 (nearest, ties to
 * even; NaN stays NaN).  Used to build the bf16 GEMM operands.
 * ------------------------------------------------------------------------ */
int o5_f32_to_bf16(size_t n, const float* src, uint16_t* dst, void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing (instrumentation for benchmarks).  The timer is
 * process-wide state and so lies outside the stateless contract of the
 * compute calls above: its records are guarded by a lock, so calls from
 * several threads do not race, but the two events of one site are paired
 * in recording order, so a site should not be timed from two streams at
 * once.
 * o5_ktimer_enable(1) clears previous records and starts recording a pair
 * of hipEvents on the caller's stream around every launch site listed
 * below; o5_ktimer_enable(0) stops recording (records are kept until the
 * next enable).  o5_ktimer_read waits for the recorded events of one site
 * and returns the summed device time in milliseconds and the number of
 * launches.  Sites: 0 lstm_fwd_gemm, 1 lstm_fwd_cell, 2 lstm_dh_gemm,
 * 3 lstm_bwd_cell, 4 lstm_dw_gemm, 5 lstm_dx_gemm, 6 ppo_loss_grad (whole
 * call), 7 adam_step, 8 gae, 9 policy_sample (whole call), 10
 * reward_process, 11 obs_normalize, 12 prelstm_fwd, 13 prelstm_bwd (whole
 * calls), 14 lstm_fwd_call (a whole o5_lstm_fwd call: one pair of events
 * for all its steps, where site 0 adds a pair around each step's launch).
 * o5_ktimer_enable_sites(mask) does the same for the sites whose bit
 * (1 << site) is set in mask (0 stops recording): every recorded pair adds
 * two event packets to the stream, so a timed run can record only the sites
 * it needs.
 * o5_ktimer_site_name returns the site's name ("" if out of range).
 * ------------------------------------------------------------------------ */
int o5_ktimer_enable(int on);
int o5_ktimer_enable_sites(unsigned int mask);
int o5_ktimer_read(int site, double* total_ms, int* launches);
const char* o5_ktimer_site_name(int site);

#ifdef __cplusplus
}
#endif

#endif /* O5_H */
