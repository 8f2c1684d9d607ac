/*
 * wm.h - C ABI of the MI355X World-Model dream library (libwm.so).
 *
 * The library runs the data-parallel hot path of RLFlow's model-based agent
 * (Parker, Alabed, Yoneki, arXiv 2205.01435):
 *   - the batched "dream" rollout of the World Model: a controller picks an
 *     action from [z_t, h_t] (section 3.4) among the valid ones (section
 *     3.1.3), an LSTM core over [z_t, one-hot a_t] updates the hidden state,
 *     and a mixture-density head samples z_{t+1} with temperature tau and
 *     predicts reward and termination (section 3.3.2; the step returns next
 *     state, reward and terminal flag as in section 3.1.1);
 *   - the teacher-forced mixture negative log-likelihood pass that fits the
 *     model (section 4.7, on random-agent data as in section 3.3.2);
 *   - a single controller decision.
 *
 * Conventions (all entry points):
 *   - Pointers are DEVICE pointers unless stated otherwise; `stream` is a
 *     hipStream_t (NULL = the default stream).  Work is enqueued on that
 *     stream and the call returns; the status covers argument checks and
 *     launch errors only.
 *   - The caller owns every buffer.  The library never allocates device
 *     memory and keeps no pointer after the call returns.  It synchronises
 *     the stream only in wm_workspace_status and under WM_FLAG_CHECK.
 *   - Matrices are row-major.  Time-major arrays are [T, B, ...].
 *   - Dimensions: B trajectories / sequences, T steps, Z latent size (a
 *     multiple of 8), H hidden size (a multiple of 16), A actions (1..2048
 *     with a one-level controller; A = N L with the two-level one, N + 1 and
 *     L at most 1024, the one-hot block of A x 4H weights under 2 GiB), K
 *     Gaussians per latent dimension (1..8).  Other values return
 *     WM_ERR_UNSUPPORTED.
 *   - Thread safety: calls may be made from several threads; calls that
 *     share output or workspace buffers must be ordered by the caller.
 *   - Random numbers: Philox4x32-10 (Salmon et al., SC'11) with key
 *     (seed & 0xffffffff, seed >> 32) and counter (block, step, traj,
 *     stream); uniform i of a stream is word i % 4 of block i / 4, mapped to
 *     ((x >> 9) + 0.5) * 2^-23.  Streams: 0 controller Gumbel noise (index
 *     = action), 1 component Gumbel noise (index = j*K + k), 2 Box-Muller
 *     uniforms (index = latent dim), 3 done uniform (index 0).
 */
#ifndef WM_H
#define WM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* hipStream_t without pulling in the HIP headers. */
typedef struct ihipStream_t *wm_stream_t;

typedef enum {
  WM_OK = 0,
  WM_ERR_INVALID_ARG = -1, /* null required pointer, bad size, tau <= 0, ...  */
  WM_ERR_UNSUPPORTED = -2, /* dims outside the compiled kernels' range        */
  WM_ERR_WORKSPACE = -3,   /* workspace smaller than wm_workspace_bytes()     */
  WM_ERR_HIP = -4          /* a HIP call or launch failed; see wm_last_error  */
} wm_status;

typedef enum {
  WM_FP32 = 0, /* fp32 weights and activations, fp32 accumulate            */
  WM_BF16 = 1  /* bf16 weights and GEMM operands (z, h), fp32 accumulate,
                  fp32 cell state and mixture arithmetic                    */
} wm_dtype;

enum {
  WM_FLAG_DONE = 1u,  /* sample the done head; else dones are 0 while live */
  WM_FLAG_TRACE = 2u, /* write h_trace / c_trace                           */
  WM_FLAG_CHECK = 4u, /* debug mode: check the device data's preconditions
                         (wm_rollout: every mask byte is 0 or 1; wm_nll,
                         wm_nll_grad: every action of a step inside its
                         sequence is in [0, A) or one of the codes -1, -2 a
                         rollout emits, every done byte is 0 or 1) with
                         device kernels that count violations in the
                         workspace's status words.  The call then waits for
                         its stream: a violation returns WM_ERR_INVALID_ARG
                         before any output is computed, and a device-side
                         failure of the computation (a barrier wait that
                         timed out) returns WM_ERR_HIP.                     */
  WM_FLAG_STEP_MASK = 8u, /* valid_mask is [T, B, A], one mask per step (the
                            valid actions depend on the state, section
                            3.1.3); else [B, A] for every step              */
  WM_FLAG_SIGMA_TAU = 16u, /* also scale the mixture's standard deviation by
                             sqrt(tau) (the temperature of Ha and
                             Schmidhuber's World Models, on which section
                             3.3 builds); without it tau acts on the
                             pi-logits only, as the paper specifies         */
  WM_FLAG_TEST_ABORT = 0x80000000u /* test support, never needed otherwise:
                            the call starts with the workspace's device
                            error word already set, as though a barrier wait
                            of the persistent kernels had timed out.  Those
                            kernels then leave at their first wait and exit
                            normally, and the status (wm_workspace_status,
                            or the return value under WM_FLAG_CHECK)
                            reports the failure whichever path ran.         */
};

typedef struct {
  int32_t Z, H, A, K;
  int32_t dtype; /* wm_dtype */
  /* Two-level controller (section 3.1.3), 0 and 0 for the one-level one: N
   * graph transformations (xfers) plus the NO-OP, each applied at one of L
   * locations.  The world model's actions are the A = N * L pairs, action
   * a = x * L + l; the controller's W_c [N+1+L, Z+H], b_c [N+1+L] hold the
   * N+1 xfer logits (row N = NO-OP) then the L location logits.          */
  int32_t N, L;
} wm_dims;

/*
 * Canonical weights, float32 device arrays (row-major [out, in]):
 *   W_g [4H, Z+A+H]  LSTM gates, rows in blocks i | f | g | o, columns
 *                    z | one-hot action | h; b_g [4H].
 *   W_m [3ZK, H]     mixture head on h_{t+1}: row p*Z*K + j*K + k holds,
 *                    for latent dim j and component k, the pi-logit (p=0),
 *                    the mean (p=1) and log sigma (p=2); b_m [3ZK].
 *   w_r [H], b_r [1] reward head on h_{t+1}.
 *   w_d [H], b_d [1] done head on h_{t+1}: P(done) = sigmoid(w_d.h + b_d).
 *   W_c [Ac, Z+H]    controller logits on [z_t, h_t] (section 3.4); b_c [Ac];
 *                    Ac = A, or N+1+L for the two-level controller.
 */
typedef struct {
  const float *W_g, *b_g;
  const float *W_m, *b_m;
  const float *w_r, *b_r;
  const float *w_d, *b_d;
  const float *W_c, *b_c;
} wm_weights;

/* Size in bytes of the packed (kernel-layout) weights for `dims`; 0 if the
 * dims are invalid or unsupported. */
size_t wm_packed_weights_bytes(const wm_dims *dims);

/* Convert canonical weights into the kernels' layout (gate-interleaved
 * rows, one-hot block transposed for column gathers, mixture rows grouped
 * per latent dimension, controller extended with the reward and done rows),
 * rounding to bf16 (nearest, ties to even) when dims->dtype is WM_BF16.
 * `packed` is a device buffer of at least wm_packed_weights_bytes(dims)
 * bytes (256-byte aligned).
 * Enqueued on `stream`; the canonical arrays may be freed once it ran. */
wm_status wm_pack_weights(const wm_dims *dims, const wm_weights *canon, void *packed,
                          size_t packed_bytes, wm_stream_t stream);

/* Workspace bytes needed by wm_rollout (which = 0), wm_nll (which = 1),
 * wm_controller_step (which = 2: it takes no workspace, so 0) or wm_nll_grad
 * (which = 3) for B rows and T steps.  0 on bad args and on sizes the call
 * refuses.  Every workspace starts with the status words that
 * wm_workspace_status reads. */
size_t wm_workspace_bytes(const wm_dims *dims, int32_t B, int32_t T, int32_t which);

/*
 * One controller decision for B states (section 3.4, masked as in section
 * 3.1.3): logits = W_c [q(z), q(h)] + b_c, where q rounds to bf16 on
 * WM_BF16 and is the identity on WM_FP32.
 *   z [B, Z], h [B, H]   float32 state.
 *   valid_mask [B, A]    uint8, nonzero = action valid.
 *   seed, step, traj0    Philox key and counter words; row b is trajectory
 *                        traj0 + b.
 *   probs [B, A]         nullable; softmax of the logits over the valid
 *                        actions (exactly 0 on invalid ones; an all-invalid
 *                        row is all 0).
 *   action [B]           int32; argmax over valid a of logits_a - ln(-ln u_a)
 *                        (a sample from `probs`), u_a uniform a of stream 0;
 *                        ties go to the lowest index; -1 if none is valid.
 * The two-level controller (dims N > 0, section 3.1.3): valid_mask holds
 * the xfer masks [B, N+1] followed by the location masks [B, N, L]; action
 * is the two-level pick described under wm_rollout (x L + l, -2 for the
 * NO-OP, -1 when nothing is valid); probs [B, N+1+L] is required and
 * receives the softmax of the valid xfers' logits, then the softmax of the
 * logits of the locations valid for the picked xfer (all 0 after a NO-OP or
 * when nothing is valid).
 */
wm_status wm_controller_step(const wm_dims *dims, const void *packed, int32_t B,
                             uint32_t traj0, const float *z, const float *h,
                             const uint8_t *valid_mask, uint64_t seed, uint32_t step,
                             float *probs, int32_t *action, wm_stream_t stream);

/*
 * B dream trajectories of T steps (sections 3.3.2 and 3.4).  Step t uses the
 * absolute step s = step0 + t and trajectory traj0 + b in its counters.  For
 * a live trajectory:
 *   1. a_t = masked Gumbel-max of the controller logits on (z_t, h_t);
 *   2. gates = W_z q(z_t) + W_h q(h_t) + W_g[:, Z + a_t] + b_g (the one-hot
 *      product is a column gather), LSTM cell -> c_{t+1} (fp32) and
 *      h_{t+1} (stored rounded to the dtype);
 *   3. mixture parameters from h_{t+1}; for each latent dim j the component
 *      k_j = argmax_k (pi_logit_jk / tau + Gumbel(stream 1, j*K + k));
 *   4. z_{t+1,j} = mu_jk + exp(log_sigma_jk) * eps_j, eps from Box-Muller on
 *      the stream-2 pair (2p, 2p+1) containing j (cos for even j, sin odd);
 *      with WM_FLAG_SIGMA_TAU, eps_j is scaled by sqrt(tau);
 *   5. reward_t = w_r.h_{t+1} + b_r; done_t = sigmoid(w_d.h_{t+1} + b_d) > u
 *      (stream 3) if WM_FLAG_DONE, else 0.
 * A done trajectory is frozen for the remaining steps: action -1, reward 0,
 * done 1, z copied, state unchanged.  A live trajectory with no valid action
 * ends at that step with the same frozen outputs.  With `lengths`, variable-
 * length trajectories are zero-padded as sequences are in section 3.3.1:
 * trajectory b is stepped for t < lengths[b]; a step t >= lengths[b] is
 * padding (action -1, reward 0, done 0, z_out[t+1] = 0) and its state stays
 * as after its last real step.
 *
 *   z0 [B, Z]            float32 initial latent.
 *   h0, c0 [B, H]        float32 initial state, nullable (= 0).
 *   done_io [B]          uint8, nullable: in = already done, out = done
 *                        after the last step.
 *   lengths [B]          int32, nullable (= T for every trajectory): the
 *                        horizon of each trajectory (values outside [0, T]
 *                        act as clamped); h_T, c_T and done_io then hold the
 *                        state after step lengths[b] - 1.
 *   valid_mask [B, A]    uint8, constant over the rollout; with
 *                        WM_FLAG_STEP_MASK [T, B, A], step t's actions
 *                        drawn from valid_mask[t].  With the two-level
 *                        controller (dims N > 0): the xfer masks [B, N+1]
 *                        followed by the location masks [B, N, L]; step 1
 *                        then picks an xfer x among the valid ones (stream 0,
 *                        index x), and for x < N a location l valid for x
 *                        (stream 4, index l), action x * L + l; x = N (the
 *                        NO-OP) ends the trajectory at that step with action
 *                        -2, reward 0, done 1 (per-step masks unsupported).
 *   tau                  mixture temperature, finite and > 0.
 *   z_out [T+1, B, Z]    float32; z_out[0] = z0.
 *   actions [T, B]       int32.   rewards [T, B] float32.   dones [T, B] uint8.
 *   h_T, c_T [B, H]      float32 final state, nullable.
 *   h_trace, c_trace [T+1, B, H]  float32 state at the start of each step and
 *                        after the last; required iff WM_FLAG_TRACE.
 *   workspace            device buffer of wm_workspace_bytes(dims, B, T, 0).
 * T = 0 is a no-op.  Results of trajectory b depend only on its own inputs,
 * traj0 + b and the weights, not on B or the other rows.
 */
wm_status wm_rollout(const wm_dims *dims, const void *packed, int32_t B, int32_t T,
                     uint32_t traj0, uint32_t step0, const float *z0, const float *h0,
                     const float *c0, uint8_t *done_io, const int32_t *lengths,
                     const uint8_t *valid_mask, uint64_t seed, float tau, uint32_t flags,
                     float *z_out, int32_t *actions, float *rewards, uint8_t *dones,
                     float *h_T, float *c_T, float *h_trace, float *c_trace, void *workspace,
                     size_t workspace_bytes, wm_stream_t stream);

/*
 * wm_rollout for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * the same call without the workspace arguments.  Its workspace is the
 * library's static device scratch, 64 MiB per GPU, held by every GPU the
 * library runs on until the process ends; a call whose rollout workspace
 * (wm_workspace_bytes(dims, B, T, 0)) is larger returns WM_ERR_UNSUPPORTED.
 * Nothing is allocated.  Every call on one GPU shares that GPU's scratch, so
 * calls that may overlap on one GPU (on different streams, or from several
 * threads without ordering) race and must be serialised by the caller.
 * wm_workspace_status does not apply (the scratch is not the caller's);
 * under WM_FLAG_CHECK the call itself reports the device status.
 */
wm_status wm_rollout_noalloc(const wm_dims *dims, const void *packed, int32_t B, int32_t T,
                             uint32_t traj0, uint32_t step0, const float *z0, const float *h0,
                             const float *c0, uint8_t *done_io, const int32_t *lengths,
                             const uint8_t *valid_mask, uint64_t seed, float tau,
                             uint32_t flags, float *z_out, int32_t *actions, float *rewards,
                             uint8_t *dones, float *h_T, float *c_T, float *h_trace,
                             float *c_trace, wm_stream_t stream);

/*
 * Teacher-forced MDN-RNN loss over B logged sequences of T steps (section
 * 4.7; padding masked as in section 3.3.1).  With h_0 = c_0 = 0:
 *   h_{t+1}, c_{t+1} = LSTM(W_z q(z_t) + W_h q(h_t) + W_g[:, Z + a_t] + b_g);
 *   loglik[t,b]    = sum_j log sum_k pi_jk N(z_{t+1,j}; mu_jk, sigma_jk)
 *                    (pi = softmax of the pi-logits, tau = 1);
 *   reward_se[t,b] = (w_r.h_{t+1} + b_r - rewards[t,b])^2;
 *   done_bce[t,b]  = softplus(rho) - dones[t,b] * rho, rho = w_d.h_{t+1} + b_d.
 *   z [T+1, B, Z] float32; actions [T, B] int32 (outside [0, A) = no action,
 *   a zero one-hot); rewards [T, B] float32; dones [T, B] uint8;
 *   lengths [B] int32 nullable (= T): steps t >= lengths[b] output 0.
 *   flags                0, or WM_FLAG_CHECK and / or WM_FLAG_TEST_ABORT.
 *   loglik, reward_se, done_bce [T, B] float32.
 *   means [3] float32 nullable: (-sum loglik / (N Z), sum se / N,
 *   sum bce / N) with N = sum of the clamped lengths (all 0 if N = 0).
 *   workspace: wm_workspace_bytes(dims, B, T, 1) bytes.
 */
wm_status wm_nll(const wm_dims *dims, const void *packed, int32_t B, int32_t T,
                 const float *z, const int32_t *actions, const float *rewards,
                 const uint8_t *dones, const int32_t *lengths, uint32_t flags, float *loglik,
                 float *reward_se, float *done_bce, float *means, void *workspace,
                 size_t workspace_bytes, wm_stream_t stream);

/*
 * Gradient of the world model's training loss (section 4.7): the sum of the
 * three means of wm_nll,
 *   L = -sum loglik / (N Z) + sum se / N + sum bce / N,
 * with respect to every world-model weight, by backpropagation through time
 * through the mixture, reward and done heads and the LSTM (the controller is
 * not part of this loss).  WM_FP32 weights only (WM_ERR_UNSUPPORTED on
 * WM_BF16).  Inputs as for wm_nll (same shapes and meanings); outputs are
 * device float32 arrays in the canonical layout of wm_weights, written
 * whole (not accumulated):
 *   loss [1] nullable; grad_W_g [4H, Z+A+H]; grad_b_g [4H];
 *   grad_W_m [3ZK, H]; grad_b_m [3ZK]; grad_w_r [H]; grad_b_r [1];
 *   grad_w_d [H]; grad_b_d [1].
 * N = 0 (all lengths 0) gives loss 0 and zero gradients.  T = 0 writes
 * nothing.  T B at most 2^22.  Every reduction runs in a fixed order: the
 * result does not depend on scheduling.  flags: as for wm_nll.
 *   workspace: wm_workspace_bytes(dims, B, T, 3) bytes, 256-byte aligned.
 */
wm_status wm_nll_grad(const wm_dims *dims, const void *packed, int32_t B, int32_t T,
                      const float *z, const int32_t *actions, const float *rewards,
                      const uint8_t *dones, const int32_t *lengths, uint32_t flags, float *loss,
                      float *grad_W_g, float *grad_b_g, float *grad_W_m, float *grad_b_m,
                      float *grad_w_r, float *grad_b_r, float *grad_w_d, float *grad_b_d,
                      void *workspace, size_t workspace_bytes, wm_stream_t stream);

/*
 * Return scan over B dreamed trajectories of T steps, for the policy updates
 * of the controller: the discounted sum of rewards that the agent maximises
 * (section 2.2) and, with a value baseline, generalised advantage estimates
 * (GAE(lambda), Schulman et al. 2016) for PPO (sections 2.3 and 4.1).  A
 * done step ends its trajectory: nothing after it is discounted into it.
 * It reads a wm_rollout's rewards and dones directly (frozen steps carry
 * reward 0 and done 1, so they add nothing).
 *   rewards [T, B] float32; dones [T, B] uint8 (nonzero = done).
 *   values [T+1, B] float32, nullable.
 *   gamma, lambda        in [0, 1]; lambda is used only with values.
 *   returns [T, B] float32:
 *     without values  G_t = r_t + gamma (1 - d_t) G_{t+1}, G_T = 0;
 *     with values     A_t + V_t, where
 *                     A_t = delta_t + gamma lambda (1 - d_t) A_{t+1}, A_T = 0,
 *                     delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t.
 *   advantages [T, B] float32, nullable; A_t (requires values).
 * B = 0 or T = 0 is a no-op.  Float arrays must be 4-byte aligned.
 */
wm_status wm_returns(int32_t B, int32_t T, const float *rewards, const uint8_t *dones,
                     const float *values, float gamma, float lambda, float *returns,
                     float *advantages, wm_stream_t stream);

/*
 * Optimiser step of the world-model training (the model is fitted on its
 * log-likelihood loss, section 4.7; the paper names no optimiser, Adam is
 * this library's reading).  In place on n fp32 parameters with their first
 * and second moments m, v (zero before step 1):
 *   m = beta1 m + (1 - beta1) g,   v = beta2 v + (1 - beta2) g^2,
 *   params -= lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps).
 * step >= 1; beta1, beta2 in [0, 1); eps > 0; lr >= 0.  Arrays 16-byte
 * aligned.  n = 0 is a no-op.
 */
wm_status wm_adam_step(int64_t n, float *params, const float *grads, float *m, float *v,
                       int32_t step, float lr, float beta1, float beta2, float eps,
                       wm_stream_t stream);

/* Host function: the learning rate at `epoch` of a second-degree polynomial
 * decay from lr0 to lr_end over `epochs` (section 4.7 decays over 5000):
 * (lr0 - lr_end) (1 - min(epoch, epochs) / epochs)^2 + lr_end. */
float wm_poly_lr(int32_t epoch, float lr0, float lr_end, int32_t epochs);

/*
 * Measurement aid (no counterpart in the paper).  While a prefix is set, every
 * kernel launch of the library whose name starts with it is bracketed by HIP
 * events on its stream.  Kernel names: "ctrl", "gates", "mdn", "init",
 * "finish", "nll_init", "nll_reduce", "nll_means", "pack", "returns", "adam", and the
 * "grad_" kernels of wm_nll_grad; "" selects all,
 * NULL turns timing off.  wm_profile_read waits for the recorded events and
 * returns the summed duration (ms) and count of the launches whose name
 * starts with `prefix` (NULL = all); wm_profile_reset forgets them.  Timing
 * adds host work per launch; leave it off outside measurement runs.
 */
wm_status wm_profile_enable(const char *prefix);
wm_status wm_profile_read(const char *prefix, double *total_ms, int64_t *launches);
wm_status wm_profile_reset(void);

/*
 * Phase timing of the persistent kernels (the small-batch fp32 rollout and
 * NLL recurrence), for measurement runs: with on != 0, each later launch of
 * those kernels stamps the device's constant-rate clock at its start, at
 * every arrival at and release from an XCD barrier, and at its end (one
 * lane per work-group; allocates a device buffer on first use and clears it
 * with an asynchronous memset per launch, so leave it off under graph
 * capture and in the no-allocation entry point; switching it on forgets the
 * last stamped launch, switching it off keeps it readable).
 * wm_profile_phases_read waits for the device and summarises the last
 * stamped launch into out[0..n)
 * (microseconds; "max" is over the 32 work-groups of an XCD, every figure
 * is then averaged over the steps and the XCDs that hold rows):
 *   out[0]  T (0: no stamped launch since wm_profile_phases)
 *   out[1]  wall time per step
 *   out[2], out[3]   0 (reserved: the controller decisions run inside the
 *                    gate phase)
 *   out[4], out[5]   gates(t) with the step's controller decisions: max
 *                    work, then its barrier (last arrival to first
 *                    release); NLL: the step's work and the barrier between
 *                    steps
 *   out[6], out[7]   mdn(t): max work, barrier
 *   out[8..10]       0, then the mean work of gates and mdn
 *   out[11], out[12] set-up before step 0 and the tail after the last step
 *                    (max work)
 * Slots 6, 7, 10 and 12 are 0 for the NLL recurrence.
 */
wm_status wm_profile_phases(int32_t on);
wm_status wm_profile_phases_read(double *out, int32_t n);

/*
 * Device-side status of the last call that used `workspace` (a workspace of
 * wm_rollout, wm_nll or wm_nll_grad), after waiting for `stream`.  The
 * persistent kernels wait for each other at barriers with a bounded spin; a
 * wait that times out (for example when other work on the device keeps some
 * of their work-groups from running) sets an error word in the workspace,
 * and every work-group then stops at its next wait, so the outputs of that
 * call are incomplete.  Returns WM_ERR_HIP if that word is set,
 * WM_ERR_INVALID_ARG if the call's WM_FLAG_CHECK pass counted violations,
 * WM_OK otherwise.  Host-side synchronisation; allocates nothing.
 */
wm_status wm_workspace_status(const void *workspace, wm_stream_t stream);

/* Text of the last non-OK status on the calling thread ("" if none). */
const char *wm_last_error(void);

/* Library version string. */
const char *wm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WM_H */
