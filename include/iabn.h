/*
 * libiabn: In-Place Activated Batch Normalization (InPlace-ABN) on AMD
 * Instinct MI355X (gfx950).
 *
 * The method: Rota Bulo, Porzi, Kontschieder, "In-Place Activated BatchNorm
 * for Memory-Optimized Training of DNNs", CVPR 2018 (arXiv:1712.02616).
 * A training-mode batch normalisation fused with a leaky ReLU that keeps only
 * its output z for the backward pass: the forward overwrites x with z
 * (Algorithm 1), and the backward recovers y = f^-1(z) and
 * xhat = (y - beta)/gamma from z, then forms the BN gradient (Algorithm 2,
 * InPlace-ABN I, with the BN backward of Sec. 3.3).  Also InPlace-ABN II,
 * and the two blocks the paper compares against (the standard block and the
 * proposed checkpointing, Sec. 3.2), on the same kernels.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are NCHW and contiguous, passed as one device pointer plus
 *    N, C and HW = H*W.  A BN unit is a channel: channel c owns the
 *    m = N*HW values x[n, c, :] (Sec. 3.1; parameters are channel-specific).
 *  - Storage type of the activation/gradient tensors: iabn_dtype_t.  All
 *    per-channel vectors (gamma, beta, running and saved statistics, dgamma,
 *    dbeta) are fp32 device arrays of length C.  Per-element arithmetic is
 *    fp32; reductions combine per-thread partial results in fp64.
 *  - The caller owns all memory.  The library never allocates, frees or
 *    synchronises; every call only enqueues kernels on `stream` (a
 *    hipStream_t; NULL is the default stream) and returns.  Results are valid
 *    once the stream has reached them.
 *  - `workspace` is caller-owned device memory of at least
 *    iabn_workspace_size(N, C, HW, dtype) bytes, 16-byte aligned.  A forward
 *    (or backward) split into its two phases must hand the same workspace,
 *    untouched, from the first phase to the second on the same stream.
 *  - Errors: every entry point validates its arguments on the host before it
 *    enqueues anything; on error it returns a nonzero iabn_status_t, changes
 *    no memory, and iabn_last_error() (per host thread) describes the cause.
 *    A failed kernel launch returns IABN_ERR_HIP.
 *  - Not checked, preconditions of the method: gamma[c] != 0 (the inversion
 *    of the scale-and-shift divides by gamma, Sec. 3.3 "Inversion of pi");
 *    gamma < 0 is allowed.  Buffers must not overlap except the documented
 *    in-place pairs.
 *  - Tensor pointers need only the alignment of their element type.  Each
 *    call reads and writes 16-byte accesses where HW and the pointers'
 *    alignment allow, else 8-, 4- or 2-byte ones (a narrower access changes
 *    the order of the sums, not the result beyond rounding).
 *  - Results are deterministic: the same inputs on the same device give
 *    bit-identical outputs (all reductions combine in a fixed order).
 *  - The library keeps no device state between calls (except the scratch
 *    of iabn_forward_train_noalloc): calls on different streams may run
 *    concurrently when they share no output or workspace.
 */
#ifndef IABN_H
#define IABN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of x / z / dz / dx. */
typedef enum {
    IABN_F32 = 0,  /* IEEE binary32 */
    IABN_F16 = 1,  /* IEEE binary16; stores round to nearest even */
    IABN_BF16 = 2  /* bfloat16; stores round to nearest even */
} iabn_dtype_t;

typedef enum {
    IABN_OK = 0,
    IABN_ERR_NULL = 1,      /* a required pointer is NULL */
    IABN_ERR_SHAPE = 2,     /* N, C or HW out of range, or N*HW < 2 in training */
    IABN_ERR_PARAM = 3,     /* eps, momentum or slope out of range */
    IABN_ERR_DTYPE = 4,     /* unknown iabn_dtype_t */
    IABN_ERR_WORKSPACE = 5, /* workspace too small or misaligned */
    IABN_ERR_HIP = 6        /* the HIP runtime rejected a launch */
} iabn_status_t;

/* Library version, major*10000 + minor*100 + patch. */
int iabn_version(void);

/* Static text for a status code. */
const char *iabn_status_string(int status);

/* Text describing the last error returned on the calling host thread. */
const char *iabn_last_error(void);

/* Bytes of workspace the training forward and the backward need for this
 * shape and storage type (the same amount for both).  Returns 0 for an
 * invalid shape or dtype. */
size_t iabn_workspace_size(int64_t N, int64_t C, int64_t HW, int dtype);

/* The entry points iabn_plan describes. */
typedef enum {
    IABN_OP_FORWARD_TRAIN = 0, /* iabn_forward_train */
    IABN_OP_BACKWARD = 1,      /* iabn_backward and iabn_backward_ii */
    IABN_OP_STD_FORWARD = 2,   /* iabn_std_forward_train */
    IABN_OP_STD_BACKWARD = 3,  /* iabn_std_backward */
    IABN_OP_CKPT_FORWARD = 4,  /* iabn_ckpt_forward_train */
    IABN_OP_CKPT_BACKWARD = 5, /* iabn_ckpt_backward */
    IABN_OP_FORWARD_EVAL = 6,  /* iabn_forward_eval */
    IABN_OP_CKPT_RECOMPUTE = 7 /* iabn_ckpt_recompute */
} iabn_op_t;

/* How an entry point runs a shape. */
typedef struct {
    int channel_resident; /* 1: one kernel, one block per channel holding the
                             channel on chip; 0: the streaming kernels (two
                             passes for the training entry points) */
    int access_bytes;     /* bytes per vector access: 16, 8, 4, 2, or the
                             element size */
    int threads;          /* threads per block */
    int reg_accesses;     /* channel-resident: accesses per thread held in
                             registers (per tensor) */
    int lds_accesses;     /* channel-resident: further accesses per thread
                             held in LDS (per tensor); any beyond are read
                             twice */
    int strips;           /* channel-resident: strip addressing (rows of
                             whole block-wide strips) */
    int xcd_order;        /* 1: blocks on each XCD take a contiguous range of
                             channels (or slices), for rows that do not end
                             on a 128-byte line */
    int64_t blocks;       /* blocks per kernel launch */
    int channels_per_block; /* channel-resident: channels per block (each
                               with threads / channels_per_block threads) */
} iabn_plan_t;

/* The kernels entry point `op` (an iabn_op_t) runs for this shape and
 * storage type when every tensor is 16-byte aligned.  The plan holds only
 * for such tensors: a tensor that is not takes narrower accesses, which can
 * change every field (the comparison blocks then take the streaming kernels,
 * InPlace-ABN's own entry points other rungs and block sizes).  Host only:
 * needs no GPU, launches nothing.  For callers that schedule around the library, and for tests of
 * the library's choices.  Validates like the entry point (shape, dtype; a
 * NULL plan is IABN_ERR_NULL, an unknown op IABN_ERR_PARAM); an empty shape
 * gives an all-zero plan. */
int iabn_plan(int op, int dtype, int64_t N, int64_t C, int64_t HW, iabn_plan_t *plan);

/*
 * Training-mode forward, Algorithm 1, in place.
 *   x_z            in: x; out: z = f(gamma * (x - mu)/sqrt(sigma^2 + eps) + beta),
 *                  with the leaky ReLU f(y) = y (y >= 0), slope*y (y < 0) of Sec. 3.3
 *                  and the per-channel batch mean mu and biased variance
 *                  sigma^2 of Sec. 3.1 (Eq. 1).
 *   gamma, beta    [C] scale and shift.
 *   running_mean, running_var
 *                  [C], updated in place:
 *                  running_mean = (1-momentum)*running_mean + momentum*mu,
 *                  running_var  = (1-momentum)*running_var + momentum*sigma^2*m/(m-1)
 *                  (the running average of minibatch statistics of Sec. 3.1,
 *                  with the unbiased variance estimate).
 *   save_mean, save_var
 *                  [C] out: mu and the biased sigma^2 (the small buffers that
 *                  Algorithm 1 keeps for the backward; only sigma^2 is needed
 *                  there).
 *   eps > 0, 0 <= momentum <= 1, slope > 0 (f must be invertible, Sec. 3.2/3.3).
 *   Requires N*HW >= 2.
 */
int iabn_forward_train(void *x_z, int dtype, const float *gamma, const float *beta,
                       float *running_mean, float *running_var, float *save_mean,
                       float *save_var, float eps, float momentum, float slope, int64_t N,
                       int64_t C, int64_t HW, void *workspace, size_t workspace_bytes,
                       void *stream);

/*
 * iabn_forward_train without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and
 * validation as iabn_forward_train; the partial results that the streaming
 * kernels keep between their two passes go to a static scratch array of
 * 128 KiB that the library holds on each device (every shape this forward
 * runs on the streaming kernels needs at most 96 KiB; a shape that needed
 * more would be rejected with IABN_ERR_WORKSPACE).  It allocates and frees
 * nothing.  The scratch of the current device is used, so `stream` must
 * belong to the current device.  All calls on one device share that
 * scratch: calls that may overlap in time on one device (different streams,
 * or host threads) race and must be ordered by the caller.
 */
int iabn_forward_train_noalloc(void *x_z, int dtype, const float *gamma, const float *beta,
                               float *running_mean, float *running_var, float *save_mean,
                               float *save_var, float eps, float momentum, float slope,
                               int64_t N, int64_t C, int64_t HW, void *stream);

/*
 * Inference-mode forward (Sec. 3.1, statistics fixed to the running
 * estimates), in place: z = f(gamma * (x - running_mean)/sqrt(running_var + eps) + beta).
 * Needs no workspace.  eps > 0, slope > 0.
 */
int iabn_forward_eval(void *x_z, int dtype, const float *gamma, const float *beta,
                      const float *running_mean, const float *running_var, float eps,
                      float slope, int64_t N, int64_t C, int64_t HW, void *stream);

/*
 * Backward, Algorithm 2 with InPlace-ABN I, in place over the gradient.
 *   z              [N,C,HW] the forward's output (read only).
 *   dz_dx          in: dL/dz; out: dL/dx.
 *   gamma, beta    [C] the forward's parameters.
 *   save_var       [C] the biased batch variance the forward saved.
 *   dgamma, dbeta  [C] out (overwritten, not accumulated):
 *                  dbeta = sum_i dy_i, dgamma = sum_i dy_i * xhat_i, where
 *                  dy = dz * f'(y), y = f^-1(z), xhat = (y - beta)/gamma.
 *   dx_i = (dy_i - dgamma*xhat_i/m - dbeta/m) * gamma/sqrt(sigma^2 + eps)  (Sec. 3.3).
 *   The derivative of f is taken from the stored z: 1 where z >= 0
 *   (including -0), slope where z < 0.
 *   eps and slope must be the forward's.  Requires N*HW >= 2.
 */
int iabn_backward(const void *z, void *dz_dx, int dtype, const float *gamma, const float *beta,
                  const float *save_var, float *dgamma, float *dbeta, float eps, float slope,
                  int64_t N, int64_t C, int64_t HW, void *workspace, size_t workspace_bytes,
                  void *stream);

/*
 * The two phases of iabn_forward_train, for callers that need to act between
 * them (timing each kernel, or combining statistics across devices).
 * iabn_forward_stats reads x and leaves per-channel partial statistics in the
 * workspace (Sec. 3.1 mean and variance, not yet combined);
 * iabn_forward_apply combines them in a fixed order, writes the statistics
 * and overwrites x with z exactly as iabn_forward_train does.  Arguments mean
 * what they mean there.
 */
int iabn_forward_stats(const void *x, int dtype, int64_t N, int64_t C, int64_t HW,
                       void *workspace, size_t workspace_bytes, void *stream);

int iabn_forward_apply(void *x_z, int dtype, const float *gamma, const float *beta,
                       float *running_mean, float *running_var, float *save_mean,
                       float *save_var, float eps, float momentum, float slope, int64_t N,
                       int64_t C, int64_t HW, void *workspace, size_t workspace_bytes,
                       void *stream);

/*
 * The two phases of iabn_backward.  iabn_backward_reduce reads z and dL/dz
 * and leaves per-channel partial sums of dy and dy*xhat (Sec. 3.3) in the
 * workspace; iabn_backward_apply combines them in a fixed order, writes
 * dgamma and dbeta and overwrites dz_dx with dL/dx exactly as iabn_backward
 * does.
 */
int iabn_backward_reduce(const void *z, const void *dz, int dtype, const float *gamma,
                         const float *beta, float slope, int64_t N, int64_t C, int64_t HW,
                         void *workspace, size_t workspace_bytes, void *stream);

int iabn_backward_apply(const void *z, void *dz_dx, int dtype, const float *gamma,
                        const float *beta, const float *save_var, float *dgamma, float *dbeta,
                        float eps, float slope, int64_t N, int64_t C, int64_t HW,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * Backward with InPlace-ABN II (Sec. 3.2 "In-Place Activated Batch
 * Normalization II" and the BN-dagger gradients of the Appendix): the same
 * arguments, outputs and in-place rule as iabn_backward, but the gradients
 * are written in terms of y = f^-1(z) instead of xhat, so the per-element
 * inversion of the scale-and-shift disappears:
 *   dbeta  = sum_i dy_i
 *   dgamma = (sum_i dy_i * y_i - beta * dbeta) / gamma
 *   dx_i   = (dy_i - dbeta/m - (y_i - beta) * dgamma/(gamma*m)) * gamma/sqrt(sigma^2 + eps).
 * Equal to iabn_backward in exact arithmetic; the rounding differs (the
 * conversion of sum dy*y cancels when |beta| >> |gamma * xhat|).
 */
int iabn_backward_ii(const void *z, void *dz_dx, int dtype, const float *gamma,
                     const float *beta, const float *save_var, float *dgamma, float *dbeta,
                     float eps, float slope, int64_t N, int64_t C, int64_t HW, void *workspace,
                     size_t workspace_bytes, void *stream);

/*
 * The standard building block of Sec. 3.2 (Fig. 2(a)), the baseline the
 * method is measured against: batch normalisation and leaky ReLU that keep
 * both the input x and the output z for the backward.
 *
 * iabn_std_forward_train: as iabn_forward_train, but out of place.
 *   x              [N,C,HW] input, read only (kept for the backward).
 *   z              [N,C,HW] out: z, the same values iabn_forward_train writes.
 *   x and z must not overlap.  Other arguments as in iabn_forward_train.
 *
 * iabn_std_backward: the BN backward from x (Sec. 3.3, xhat = (x - mu)/sqrt(sigma^2 + eps))
 * and the activation's backward from z (dy = dz * f'(y), f' from the sign of
 * z as in iabn_backward).
 *   x, z           [N,C,HW] the forward's input and output (read only).
 *   dz_dx          in: dL/dz; out: dL/dx (in place).
 *   save_mean, save_var
 *                  [C] the batch mean and biased variance the forward saved.
 *   dgamma, dbeta  [C] out, overwritten: dbeta = sum dy, dgamma = sum dy*xhat;
 *   dx as in iabn_backward.  x, z and dz_dx must not overlap.
 */
int iabn_std_forward_train(const void *x, void *z, int dtype, const float *gamma,
                           const float *beta, float *running_mean, float *running_var,
                           float *save_mean, float *save_var, float eps, float momentum,
                           float slope, int64_t N, int64_t C, int64_t HW, void *workspace,
                           size_t workspace_bytes, void *stream);

int iabn_std_backward(const void *x, const void *z, void *dz_dx, int dtype, const float *gamma,
                      const float *beta, const float *save_mean, const float *save_var,
                      float *dgamma, float *dbeta, float eps, float slope, int64_t N, int64_t C,
                      int64_t HW, void *workspace, size_t workspace_bytes, void *stream);

/*
 * The proposed checkpointing of Sec. 3.2 (Fig. 2(c)): the forward keeps only
 * the normalised xhat; the backward recomputes z = f(gamma*xhat + beta) for
 * the layers that need it and runs the BN backward from the stored xhat
 * (BN*, which skips the normalisation step).
 *
 * iabn_ckpt_forward_train: statistics and running estimates as
 * iabn_forward_train.
 *   x_xhat         in: x; out: xhat = (x - mu)/sqrt(sigma^2 + eps), rounded to the
 *                  storage type.
 *   z              [N,C,HW] out: z = f(gamma*xhat + beta), formed from xhat as
 *                  stored (so iabn_ckpt_recompute reproduces it bit for bit).
 *   x_xhat and z must not overlap.
 *
 * iabn_ckpt_recompute: z = f(gamma*xhat + beta) from the stored xhat, out of
 * place (xhat and z must not overlap).  No workspace, no statistics; slope > 0.
 *
 * iabn_ckpt_backward: the BN backward from the stored xhat; f' is taken from
 * the sign of y = gamma*xhat + beta (one fused multiply-add, so the sign is
 * that of the exact value; 0 takes the identity side).
 *   xhat           [N,C,HW] read only.
 *   dz_dx          in: dL/dz; out: dL/dx (in place).
 *   save_var, dgamma, dbeta, eps, slope as in iabn_backward; dbeta = sum dy,
 *   dgamma = sum dy*xhat, dx as in iabn_backward.
 */
int iabn_ckpt_forward_train(void *x_xhat, void *z, int dtype, const float *gamma,
                            const float *beta, float *running_mean, float *running_var,
                            float *save_mean, float *save_var, float eps, float momentum,
                            float slope, int64_t N, int64_t C, int64_t HW, void *workspace,
                            size_t workspace_bytes, void *stream);

int iabn_ckpt_recompute(const void *xhat, void *z, int dtype, const float *gamma,
                        const float *beta, float slope, int64_t N, int64_t C, int64_t HW,
                        void *stream);

int iabn_ckpt_backward(const void *xhat, void *dz_dx, int dtype, const float *gamma,
                       const float *beta, const float *save_var, float *dgamma, float *dbeta,
                       float eps, float slope, int64_t N, int64_t C, int64_t HW,
                       void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* IABN_H */
