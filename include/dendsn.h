/*
 * dendsn.h — C ABI of the DendSN layer scan on AMD Instinct MI355X (gfx950).
 *
 * The library computes one layer of dendritic spiking neurons (DendSN) over T
 * time steps and the surrogate-gradient backpropagation through time of the
 * same layer, as defined in "Scalable Dendritic Modeling Advances Expressive
 * and Robust Deep Spiking Neural Networks" (Huang et al., arXiv 2412.06355):
 *
 *   Methods, "Dendritic spiking neuron":
 *     Eq. (methods-compartment)        Vd_i[t] = alpha Vd_i[t-1] + X_i[t],  Vd[0] = 0
 *     Eq. (methods-branch-aggregation) Y_b[t]  = psi(||Vd_{C_b}[t] - xi_{C_b}|| / zeta_b), the L2 norm
 *                                      over the KC = comps_per_branch compartments of branch b
 *     Eq. (methods-mexican-hat)        psi(x)  = (1 - x^2) exp(-x^2/2), or psi(x) = x
 *     Eq. (methods-soma-input)         Z[t]    = sum_b kappa_b Y_b[t]
 *     Eq. (methods-lif-reset-charge)   H[t]    = beta (1 - S[t-1]) H[t-1] + Z[t],  H[0] = S[0] = 0
 *     Eq. (methods-lif-fire)           S[t]    = 1 if H[t] - v_th >= 0 else 0
 *   Methods, "DendSN variants": Stateless Dendrite (Vd_b[t] = X_b[t]) and the
 *     residual dendrite, Eq. (methods-residual): Z[t] += (1/P) sum_i X_i[t]
 *     (ResStateful / ResStateless).
 *   Methods, "Dendritic spiking neuron", soma: a LIF soma with a fixed decay, or
 *     the parametric LIF (PLIF) soma, whose decay beta is learnable.
 *   Methods, "Dendritic branch gating": kappa* = kappa (.) m with a fixed binary
 *     mask m per task, Eq. (methods-dbg-mask) and Eq. (methods-dbg-sampling).
 *   Methods, "Dendritic spiking neural networks": layer form — neurons of one
 *     channel share xi, zeta, kappa; alpha is shared by the whole layer; the
 *     backward replaces Theta' by a surrogate derivative, Eq. (methods-sg).
 *
 * Layout (all row-major), with P = B * KC compartments per neuron:
 *   X, grad_x          [T, N, P]  compartments innermost, I/O dtype (fp32 or bf16); compartment
 *                                 i lies on branch i / KC (a branch's compartments are adjacent)
 *                      or, with cfg->layout = DENDSN_LAYOUT_CHANNEL_MAJOR, [T, batch, C, P, S]:
 *                                 the paper's layer layout (Methods, "Dendritic spiking neural
 *                                 networks"), where the producing layer's C*P channels are cut
 *                                 into groups of P consecutive feature maps, one group per
 *                                 output channel (the same memory as [T, N, P] when S = 1)
 *   spikes, grad_spikes[T, N]     I/O dtype; spikes are exactly 0.0 or 1.0
 *   v_soma, grad_v_soma[T, N]     fp32; v_soma[t] = H[t], the potential before the reset
 *   kappa, zeta        [C, B]     fp32 per-channel branch parameters
 *   xi                 [C, P]     fp32 per-channel compartment translations
 *   mask               [C, B]     uint8, nonzero = branch kept
 *   alpha              [1]        fp32 on the device (a learnable layer scalar)
 *   beta               [1]        fp32 on the device, optional: a learnable somatic decay
 *                                 (PLIF); NULL uses cfg->beta
 *   Neuron n = (b_idx * C + c) * S + s for batch item b_idx, channel c, spatial
 *   position s; a fully connected layer has S = 1.
 *
 * Conventions:
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  The library
 *     allocates nothing, keeps no state between calls (the scratch array of
 *     dendsn_backward_noalloc aside) and never synchronises: every call enqueues
 *     kernels on the given stream and returns.
 *   - X, grad_x, ckpt and workspace must be 16-byte aligned; every other tensor
 *     must be aligned to its element size.
 *   - Outputs are overwritten, never accumulated.
 *   - Every argument check runs on the host before anything is launched.  On
 *     failure the call returns a status, writes nothing, and a description of the
 *     first failed check is available from dendsn_last_error() on the calling
 *     thread.  A failed launch returns DENDSN_E_HIP.  Faults inside a kernel
 *     surface at the caller's next synchronisation.
 *   - An empty layer (T, batch, C or S of 0) is valid: dendsn_forward has no
 *     output element to write and launches nothing; dendsn_backward (and
 *     dendsn_backward_noalloc) write +0 to every parameter gradient requested,
 *     the value of a sum with no terms.  Pointers to arrays of no elements may
 *     be NULL there (x, spikes, grad_spikes, grad_x; kappa when C = 0);
 *     dendsn_ckpt_bytes is 0 and dendsn_bwd_workspace_bytes stays positive.
 *   - Size limits, refused with DENDSN_E_UNSUPPORTED: one sample's slice of X
 *     (C * S * P elements) must stay below 4 GiB, since lanes address it with
 *     32-bit byte offsets (whole tensors may be larger); the grid must stay below
 *     2^31 blocks.  Counts beyond 2^46 elements (N, or T * N * P) are refused
 *     with DENDSN_E_INVALID.
 *   - Not checked (it would need a device synchronisation): zeta > 0,
 *     0 <= alpha < 1, finite inputs, and that pointers address device memory of
 *     the stated size.
 */
#ifndef DENDSN_H
#define DENDSN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dendsn_status {
    DENDSN_OK = 0,
    DENDSN_E_INVALID = 1,      /* an argument violates the contract            */
    DENDSN_E_UNSUPPORTED = 2,  /* valid model, but a shape no compiled kernel covers */
    DENDSN_E_WORKSPACE = 3,    /* workspace missing or smaller than required    */
    DENDSN_E_HIP = 4           /* a kernel launch failed                        */
} dendsn_status;

typedef enum dendsn_io { DENDSN_IO_F32 = 0, DENDSN_IO_BF16 = 1 } dendsn_io;
typedef enum dendsn_psi { DENDSN_PSI_IDENTITY = 0, DENDSN_PSI_MEXHAT = 1 } dendsn_psi;
typedef enum dendsn_sg { DENDSN_SG_ATAN = 0, DENDSN_SG_SIGMOID = 1 } dendsn_sg;
typedef enum dendsn_layout { DENDSN_LAYOUT_NPB = 0, DENDSN_LAYOUT_CHANNEL_MAJOR = 1 } dendsn_layout;

typedef struct dendsn_cfg {
    int64_t T;                 /* time steps, >= 0 (0: an empty layer)                     */
    int64_t batch;             /* batch items, >= 0                                        */
    int64_t C;                 /* channels (parameter sets), >= 0                          */
    int64_t S;                 /* spatial positions per channel, >= 0 (1 = fully connected)*/
    int32_t B;                 /* branches per neuron, 1..128                              */
    int32_t comps_per_branch;  /* compartments per branch KC = P / B: 1, 2 or 4            */
    int32_t stateful;          /* 1: leaky compartments; 0: Stateless Dendrite             */
    int32_t detach_reset;      /* 1: no gradient through the reset factor (1 - S[t-1])     */
    int32_t ckpt_every;        /* K >= 1: state checkpoint after every K steps (K >= T: none) */
    int32_t io;                /* dendsn_io: storage of X, spikes, grad_x, grad_spikes     */
    int32_t psi;               /* dendsn_psi: dendritic activation                          */
    int32_t sg;                /* dendsn_sg: surrogate derivative used by the backward      */
    float sg_scale;            /* slope a of the sigmoid surrogate sigma(a x); > 0          */
    float beta;                /* somatic decay, 0 <= beta < 1                              */
    float v_th;                /* firing threshold (the paper uses 1)                       */
    int32_t batch_groups;      /* tuning: batch groups per launch, 0 = automatic           */
    int32_t residual;          /* 1: residual dendrite, Z += mean of the neuron's inputs   */
    int32_t layout;            /* dendsn_layout of X and grad_x                            */
} dendsn_cfg;

/*
 * Size in bytes of the state-checkpoint buffer that dendsn_forward fills and
 * dendsn_backward reads: gradient checkpointing of the dendritic integration
 * (Results, DendSNN efficiency paragraph: the backward recomputes the dendrite
 * instead of storing it).  nck = ceil(T / K) - 1 checkpoints, the states after
 * steps K, 2K, ... < T: nck * N * (P + 1) * 4 bytes for a stateful dendrite (the
 * P compartment states and the somatic potential), nck * N * 4 for the
 * Stateless Dendrite (only the somatic potential: its compartment state is the
 * input itself).  Zero when K >= T or the layer is empty.  Returns
 * DENDSN_E_INVALID / _UNSUPPORTED for a bad cfg.
 */
dendsn_status dendsn_ckpt_bytes(const dendsn_cfg* cfg, size_t* bytes);

/*
 * Size in bytes of the scratch workspace dendsn_backward needs for its
 * per-block parameter-gradient partials (always > 0).  It depends on the whole
 * cfg, including batch_groups.
 */
dendsn_status dendsn_bwd_workspace_bytes(const dendsn_cfg* cfg, size_t* bytes);

/*
 * Forward scan over t = 1..T (equations above).
 *   x       [T,N,P] io    required
 *   alpha   [1] fp32      required when cfg->stateful, ignored otherwise
 *   beta    [1] fp32      optional learnable somatic decay (NULL: cfg->beta)
 *   kappa   [C,B] fp32    required (for dendritic branch gating with per-task dense
 *                         strengths, DBG_e, pass the task's own [C,B] table)
 *   xi      [C,P] fp32    NULL means 0
 *   zeta    [C,B] fp32    NULL means 1
 *   mask    [C,B] uint8   NULL means every branch kept
 *   spikes  [T,N] io      required output
 *   v_soma  [T,N] fp32    optional output (NULL: not written)
 *   ckpt    dendsn_ckpt_bytes bytes, optional output; NULL is allowed only for
 *           inference (no backward will follow), or when K >= T.
 */
dendsn_status dendsn_forward(const dendsn_cfg* cfg, const void* x, const float* alpha,
                             const float* beta, const float* kappa, const float* xi,
                             const float* zeta, const uint8_t* mask, void* spikes, float* v_soma,
                             float* ckpt, hipStream_t stream);

/*
 * Backward scan: gradients of  sum(grad_spikes * S) + sum(grad_v_soma * H)  with
 * Theta'(H - v_th) replaced by the surrogate cfg->sg, through time (BPTT).
 * The dendrite is recomputed from x and the checkpoints (gradient
 * checkpointing of the dendritic integration; Results, DendSNN efficiency
 * paragraph); nothing else of the forward is stored.  The call must use the
 * same cfg, x, alpha, beta, kappa, xi, zeta and mask as the forward that wrote ckpt.
 *   ckpt         required when nck > 0 (see dendsn_ckpt_bytes)
 *   grad_spikes  [T,N] io     required
 *   grad_v_soma  [T,N] fp32   NULL means 0
 *   grad_x       [T,N,P] io   required output (with the residual dendrite it includes the
 *                dH/P of the residual path, also on gated-off branches)
 *   grad_alpha   [1] fp32     optional output (0 for the Stateless Dendrite)
 *   grad_beta    [1] fp32     optional output: d/d beta of the loss (PLIF soma), summed
 *                over time and neurons; meaningful whether beta came from cfg or the device
 *   grad_kappa, grad_zeta [C,B], grad_xi [C,P]  fp32 optional outputs, summed over
 *                time, batch and spatial positions; exactly 0 for gated-off branches.
 *   workspace    device scratch of at least dendsn_bwd_workspace_bytes bytes,
 *                clobbered by the call.
 * Results are deterministic: the same inputs give bit-identical outputs.
 */
dendsn_status dendsn_backward(const dendsn_cfg* cfg, const void* x, const float* alpha,
                              const float* beta, const float* kappa, const float* xi,
                              const float* zeta, const uint8_t* mask, const float* ckpt,
                              const void* grad_spikes, const float* grad_v_soma, void* grad_x,
                              float* grad_alpha, float* grad_beta, float* grad_kappa,
                              float* grad_xi, float* grad_zeta, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/*
 * Maximum workspace of dendsn_backward_noalloc: 32 MiB of device memory per
 * GPU, held by the library from the first call on that GPU until the process
 * ends (every benchmark-sized layer needs at most 25.2 MiB).
 */
#define DENDSN_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/*
 * dendsn_backward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, outputs and bit-identical results, without a workspace.
 * The parameter-gradient partials go to a scratch array of
 * DENDSN_NOALLOC_SCRATCH_BYTES that the library keeps in each GPU's memory;
 * nothing is allocated by the call.  The call runs on the current device, and
 * `stream` must belong to it (else DENDSN_E_INVALID).
 *   - A layer whose dendsn_bwd_workspace_bytes exceeds the scratch size is
 *     refused with DENDSN_E_WORKSPACE before anything is launched.
 *   - Every call on one GPU shares that GPU's scratch array.  Calls that may
 *     overlap on one GPU (several streams or host threads) race on it: the
 *     caller serialises them.  Each call writes every scratch byte it reads, so
 *     what an earlier call left there does not matter.
 */
dendsn_status dendsn_backward_noalloc(const dendsn_cfg* cfg, const void* x, const float* alpha,
                                      const float* beta, const float* kappa, const float* xi,
                                      const float* zeta, const uint8_t* mask, const float* ckpt,
                                      const void* grad_spikes, const float* grad_v_soma,
                                      void* grad_x, float* grad_alpha, float* grad_beta,
                                      float* grad_kappa, float* grad_xi, float* grad_zeta,
                                      hipStream_t stream);

/* Static name of a status code. */
const char* dendsn_status_str(dendsn_status status);

/* Description of the last failed check on the calling thread ("" if none). */
const char* dendsn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DENDSN_H */
