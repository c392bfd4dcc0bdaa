/*
 * fewbit.h -- C ABI of the few-bit activation library for AMD MI355X (gfx950).
 *
 * Method: "Few-Bit Backward: Quantized Gradients of Activation Functions for
 * Memory Footprint Reduction" (Novikov et al., ICML 2022).  A pointwise
 * activation y = f(x) keeps for its backward pass only the index of the
 * interval of a piecewise-constant approximation q of f' that each input
 * falls in (Sec. 2, Eq. (2)); the backward multiplies the incoming gradient
 * by the stored interval value (Eq. (1) with f' replaced by q; Listing 1).
 * The approximation minimises the weighted L2 error of Eq. (3) and is found
 * once per activation by a dynamic programme over a grid (Sec. 3,
 * Eqs. (6)-(9)).
 *
 * Conventions for every entry point:
 *   - Plain C types only.  Device pointers are HIP device addresses; the
 *     stream argument is a hipStream_t passed as void* (NULL = null stream).
 *   - Device: the current HIP device must own the buffers and the stream;
 *     fwd / bwd reject a stream of another device with FEWBIT_E_INVALID.
 *   - The caller owns every buffer.  The library never allocates or frees
 *     device memory and never synchronises the caller's streams.
 *   - All argument checks run on the host before anything is launched, so a
 *     call that returns an error has written nothing.  Asynchronous device
 *     faults surface at the caller's next synchronisation.
 *   - Global state: the compute-unit count of each device, read once (it
 *     sizes the launch grid).  The library keeps no device memory of its
 *     own: the fp16 / bf16 forward builds its lookup tables in every
 *     workgroup's LDS.  No call synchronises anything, so every call,
 *     including a process's first, may be captured into a graph.  Calls are
 *     reentrant and thread-safe.
 *   - No C++ exception crosses this interface.
 */
#ifndef FEWBIT_H
#define FEWBIT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ */
/* Status codes (returned as int; 0 = success).                        */
/* ------------------------------------------------------------------ */
#define FEWBIT_OK           0
#define FEWBIT_E_INVALID   -1  /* bad size / enum / flag / weight          */
#define FEWBIT_E_NULL      -2  /* NULL pointer with n > 0                  */
#define FEWBIT_E_ALIGN     -3  /* pointer not 16-byte aligned              */
#define FEWBIT_E_DTYPE     -4  /* unknown storage type                     */
#define FEWBIT_E_BITS      -5  /* bits outside 1..4                        */
#define FEWBIT_E_NOMEM     -6  /* host allocation failed (fit only)        */
#define FEWBIT_E_NUMERIC   -7  /* table not strictly sorted / not finite   */
#define FEWBIT_E_HIP       -8  /* a HIP launch or runtime call failed      */

/* Activations: the rows of Table 1 (Swish is x*sigmoid(x), Sec. 4). */
#define FEWBIT_GELU     0      /* x * Phi(x), Phi the standard normal cdf  */
#define FEWBIT_SILU     1      /* x * sigmoid(x)                           */
#define FEWBIT_SIGMOID  2      /* 1 / (1 + exp(-x))                        */
#define FEWBIT_TANH     3      /* tanh(x)                                  */
#define FEWBIT_RELU     4      /* max(x, 0); f' = 1 for x > 0, else 0      */
#define FEWBIT_SELU     5      /* lambda x (x > 0), lambda alpha (e^x - 1)
                                  (x <= 0), lambda = 1.0507009873554805,
                                  alpha = 1.6732632423543772              */
#define FEWBIT_SOFTPLUS 6      /* log(1 + e^x)                             */

/* Storage types of x, y, grad_out, grad_in. */
#define FEWBIT_F32   0         /* IEEE binary32                            */
#define FEWBIT_F16   1         /* IEEE binary16                            */
#define FEWBIT_BF16  2         /* bfloat16 (upper half of a binary32)      */

/* Weight kinds for the fit (Sec. 3, Eq. (3)); w = 0 outside [A, B]. */
#define FEWBIT_W_UNIFORM  0    /* w(x) = 1 on [A, B] (not normalised)      */
#define FEWBIT_W_NORMAL   1    /* density of N(mu, sigma^2)                */
#define FEWBIT_W_MIXTURE  2    /* (1-p) N(mu, sigma^2) + p N(mu, sigma2^2) */

/* Table flags. */
#define FEWBIT_FLAG_SYMMETRIC 1 /* even f': bins apply to |x|, fit on [0,B]
                                   (Fig. 3 caption)                        */
/* Fit flag (fewbit_fit_table only; never set in a table). */
#define FEWBIT_FLAG_REFINE    2 /* refine the DP boundaries by gradient
                                   descent on L(s, y(s)) (Sec. 3)          */
/* Kernel choice of the fp16 / bf16 forward (may be set in a table by the
 * caller; at most one of the two; ignored by fp32 forwards and by the
 * backward).  Without either, fewbit_fwd picks by size (see
 * fewbit_fwd16_table_min).  Both kernels give results within the same
 * bounds; these flags only choose how the work is done. */
#define FEWBIT_FLAG_TABLE_FWD   4  /* table kernel at every size           */
#define FEWBIT_FLAG_ELEMENT_FWD 8  /* per-element kernel at every size     */

typedef struct fewbit_weight {
    int32_t kind;          /* FEWBIT_W_*                                   */
    int32_t reserved;      /* must be 0                                    */
    double A, B;           /* support, A < B, both finite                  */
    double mu, sigma;      /* normal / mixture core, sigma > 0             */
    double p, sigma2;      /* mixture weight 0 <= p <= 1 and second sigma  */
} fewbit_weight;

/*
 * A fitted approximation q(x | s, v) of f' (Eq. (2)), K = 2^bits intervals.
 *   s[0..K-2]  interior boundaries, strictly increasing, finite (fp32).
 *              Interval m is [s[m-1], s[m]) with s[-1] = -inf and
 *              s[K-1] = +inf: the outer intervals are unbounded.
 *              Unused slots hold +inf.
 *   v[0..K-1]  interval values (fp32, finite).  Unused slots hold 0.
 *   loss       the minimised L of Eq. (3) (doubled for FLAG_SYMMETRIC).
 * The table is a host object; fwd/bwd copy it into kernel arguments at the
 * call, so it may be reused or freed as soon as the call returns.
 */
typedef struct fewbit_table {
    int32_t act;           /* FEWBIT_GELU .. FEWBIT_SOFTPLUS               */
    int32_t bits;          /* 1..4                                         */
    int32_t flags;         /* FEWBIT_FLAG_SYMMETRIC, FEWBIT_FLAG_TABLE_FWD,
                              FEWBIT_FLAG_ELEMENT_FWD                      */
    int32_t reserved;      /* must be 0                                    */
    float s[15];
    float v[16];
    double loss;
} fewbit_table;

/*
 * fewbit_fit_table -- optimal piecewise-constant fit of f' (Sec. 3).
 *
 * Minimises Eq. (3) over boundaries and values by the discretised dynamic
 * programme of Eq. (7) on the uniform grid t_i = A + i (B-A)/n_grid,
 * i = 0..n_grid, with the O(n) prefix integrals of Eqs. (8)-(9) evaluated
 * by 8-point Gauss-Legendre quadrature per cell; every interval spans at
 * least one cell.  Values follow Eq. (4).  With FEWBIT_FLAG_SYMMETRIC the
 * fit is made on [max(A,0), B] for |x| and the reported loss is doubled.
 * With FEWBIT_FLAG_REFINE the DP boundaries are then moved off the grid by
 * steepest descent on L(s, y(s)) with its analytic gradient (Sec. 3),
 * backtracking so that every step lowers L and keeps the boundaries sorted
 * inside (A, B); integrals at off-grid points are the grid prefix plus the
 * partial cell by the same rule.  The output table's flags keep only
 * FEWBIT_FLAG_SYMMETRIC.
 * Runs on the host only; O(n_grid^2 * 2^bits) time, O(n_grid * 2^bits)
 * memory.  Deterministic.
 *
 *   act, bits          as in fewbit_table (bits 1..4)
 *   flags              FEWBIT_FLAG_SYMMETRIC and / or FEWBIT_FLAG_REFINE
 *   w                  weight function and support (host pointer)
 *   n_grid             number of grid cells, 2^bits <= n_grid <= 2^20
 *   out                receives the table (host pointer)
 * Returns FEWBIT_OK, FEWBIT_E_INVALID / _BITS / _NULL for bad arguments,
 * FEWBIT_E_NOMEM, or FEWBIT_E_NUMERIC if the fp32 boundaries collapse.
 */
int fewbit_fit_table(int32_t act, int32_t bits, const fewbit_weight* w,
                     int64_t n_grid, int32_t flags, fewbit_table* out);

/* Number of uint32 words holding n codes of `bits` bits: ceil(n*bits/32).
 * This is the storage the method keeps for the backward pass instead of x:
 * log2(k) bits per element for a k-interval approximation (Sec. 2, the
 * compression ratio stated after Eq. (2)), packed into whole words.
 * Returns -1 for n < 0 or bits outside 1..4. */
int64_t fewbit_packed_words(int64_t n, int32_t bits);

/*
 * fewbit_fwd -- forward of the few-bit activation (Listing 1, forward).
 *
 *   y[i]    = f(x[i]) evaluated in fp32 and rounded to nearest even in the
 *             storage type (same shape and layout as x, flat contiguous).
 *   idx[i]  = number of boundaries s[m] <= x[i] (of |x[i]| with the
 *             symmetric flag), 0..K-1: half-open intervals, NaN -> 0.
 *   codes   = the idx stream, bits per element, packed densely little-endian
 *             LSB-first: bit t of idx[i] is stream bit p = bits*i + t, kept
 *             in codes[p / 32] at bit p % 32.  Exactly
 *             fewbit_packed_words(n, bits) words are written; unused high
 *             bits of the last word are written as zero.
 *
 *   t      host pointer to the table (act, bits, flags taken from it)
 *   dtype  FEWBIT_F32 / FEWBIT_F16 / FEWBIT_BF16
 *   x, y   device pointers to n elements, 16-byte aligned; y == x (in place)
 *          is allowed, any other overlap is undefined
 *   codes  device pointer, 16-byte aligned, fewbit_packed_words(n, bits)
 *          words; must not overlap x or y
 *   n      element count >= 0 (0 is a no-op)
 *   stream hipStream_t (as void*), the launch is asynchronous on it
 */
int fewbit_fwd(const fewbit_table* t, int32_t dtype, const void* x, void* y,
               uint32_t* codes, int64_t n, void* stream);

/* Which of the two fp16 / bf16 forward kernels fewbit_fwd runs: from the
 * returned element count on, the table kernel (outputs and interval indices
 * looked up per input bit pattern in tables each workgroup builds in LDS);
 * below it, the per-element kernel (f and the compares evaluated for every
 * element).  The count depends on the activation, the bit width and the
 * type (dtype FEWBIT_F16 or FEWBIT_BF16); INT64_MAX where the per-element
 * kernel runs at every size.  Both kernels give results within the same
 * bounds: indices and codes identical, y within one unit in the last place
 * of the correctly rounded f.  This only tells a caller (or a test) which
 * kernel a given n reaches.  Returns -1 for an unknown activation, bits
 * outside 1..4, or another type.  Host only, no device access.  (A query of
 * the library's dispatch, not an operation of the paper.) */
int64_t fewbit_fwd16_table_min(int32_t act, int32_t bits, int32_t dtype);

/*
 * fewbit_bwd -- backward of the few-bit activation (Eq. (1) with f'(x)
 * replaced by q(x); Listing 1, backward).
 *
 *   grad_in[i] = round_dtype( fp32( float(grad_out[i]) * v[idx[i]] ) )
 *
 * i.e. the product is formed in fp32 and then rounded to nearest even in the
 * storage type (two roundings for fp16 / bf16, one for fp32).
 *
 *   t         host pointer to the same table the forward used
 *   dtype     storage type of grad_out and grad_in
 *   grad_out  device pointer, n elements, 16-byte aligned
 *   codes     device pointer written by fewbit_fwd for the same n, 16-byte
 *             aligned
 *   grad_in   device pointer, n elements, 16-byte aligned; grad_in ==
 *             grad_out is allowed, any other overlap is undefined
 *   n, stream as for fewbit_fwd
 */
int fewbit_bwd(const fewbit_table* t, int32_t dtype, const void* grad_out,
               const uint32_t* codes, void* grad_in, int64_t n, void* stream);

/* Static description of a status code (never NULL).  Error reporting of
 * this interface, not an operation of the paper. */
const char* fewbit_strerror(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* FEWBIT_H */
