/*
 * qlayer.h -- C ABI of the batched quantum-layer library (HIP, gfx950).
 *
 * The library simulates a batch of parameterised quantum circuits on one
 * GPU and returns what the paper's quantum node hands to the rest of a hybrid
 * network (Sec. "Quantum Node"): the measured outputs in the forward pass and,
 * for back-propagation (Sec. "Optimization", hybrid optimisation), the
 * gradient of the loss with respect to the circuit parameters. The quantum
 * node's backward returns the gradient multiplied by the upstream gradient
 * (appendix, hybrid quantum-classical network, class Hybrid), i.e. a
 * vector-Jacobian product. The angles of the rotation gates are bound either
 * to input features (angle encoding, Sec. "Quantum Data") or to trainable
 * weights shared by every sample of the batch.
 *
 * Conventions
 *   - qubit q is bit q of the amplitude index; the initial state is |0...0>;
 *   - H = [[1,1],[1,-1]]/sqrt(2); RX(t), RY(t), RZ(t) = exp(-i t P / 2) for
 *     P = X, Y, Z; CNOT(q0 = control, q1 = target); CZ(q0, q1);
 *   - expz[b][i] is the exact expectation <Z_i> of sample b (the limit of
 *     infinitely many measurement shots), no renormalisation;
 *   - grad_inputs[b][f]  = sum_i grad_out[b][i] d expz[b][i] / d inputs[b][f]
 *     grad_weights[p]    = sum_b sum_i grad_out[b][i] d expz[b][i] / d weights[p]
 *     (every occurrence of an input or weight in the gate list adds up);
 *   - gradients are computed by adjoint differentiation (one reverse sweep
 *     that un-applies the gates and accumulates Im<lambda|P|psi> per rotation).
 *
 * Precision: QL_C64 states are complex64 (fp32 real/imag), angles, grad_out
 * and all outputs are fp32; QL_C128 uses complex128 and fp64 throughout.
 * Every reduction runs in a fixed order, so results are bit-reproducible run
 * to run. For QL_C64, sums over one wavefront and over the tiles of one
 * workgroup are fp32; sums across wavefronts, workgroups and the batch are
 * fp64.
 *
 * Memory: all array arguments of ql_forward / ql_forward_backward are DEVICE
 * pointers on the current HIP device, row-major and contiguous, owned by the
 * caller. The caller also provides the device workspace (size from
 * ql_workspace_bytes). The library never allocates device memory in these
 * calls; it only writes the workspace and the outputs. (The first call of
 * each dtype on a handle makes a pinned host copy of the handle's plan tables,
 * which later calls upload by DMA; ql_circuit_destroy waits, through an event
 * per stream that uploaded from it, for the last such upload on each of those
 * streams before freeing it.) Outputs are
 * overwritten (not accumulated). Buffers must not alias each other or the
 * workspace.
 *
 * Errors: every function returns QL_OK (0) or a negative QL_E* code and sets a
 * thread-local message readable with ql_last_error(). All argument checks
 * happen before anything is launched. Calls are asynchronous on the given
 * stream; results are valid once the stream has been synchronised. A circuit
 * handle is immutable after creation and may be used from several threads and
 * streams at once, each with its own workspace.
 */
#ifndef QLAYER_H
#define QLAYER_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Gate kinds.
 *
 * QL_CRX/QL_CRY/QL_CRZ (q0 = control, q1 = target): the rotation of the
 * target on the amplitudes whose control bit is 1, |0><0| (x) I + |1><1| (x)
 * R(t) -- the controlled rotations of the paper's quantum autoencoder
 * (appendix "Quantum Autoencoder"). Their gradient is exact (generator
 * |1><1| (x) P).
 *
 * QL_PAULI (q0, q1 = -1, src = QL_SRC_INPUT): one quantum trajectory of a
 * Pauli channel, the noise model of the paper's noise-inclusive simulator
 * (Sec. "Unification of Classical and Quantum Machine"). With the channel's
 * probabilities (p_x, p_y, p_z) (ql_circuit_desc.pauli_p) and the sample's
 * uniform u = inputs[b][index] in [0, 1), it applies X if u < p_x, else Y if
 * u < p_x + p_y, else Z if u < p_x + p_y + p_z, else nothing (fp64 sums in that
 * order). The mean of <Z> over samples with independent uniforms estimates
 * the noisy expectation; the uniform gets no gradient. */
enum { QL_H = 0, QL_RX = 1, QL_RY = 2, QL_RZ = 3, QL_CNOT = 4, QL_CZ = 5,
       QL_CRX = 6, QL_CRY = 7, QL_CRZ = 8, QL_PAULI = 9 };

/* Where a rotation angle comes from: H/CNOT/CZ use QL_SRC_NONE; RX/RY/RZ and
 * the controlled rotations use QL_SRC_INPUT (feature `index` of each sample)
 * or QL_SRC_WEIGHT (trainable weight `index`). */
enum { QL_SRC_NONE = 0, QL_SRC_INPUT = 1, QL_SRC_WEIGHT = 2 };

/* One gate. One-qubit gates use q0 and set q1 = -1. */
typedef struct {
    int32_t kind, q0, q1, src, index;
} ql_gate;

/* Initial-state embeddings (Sec. "Quantum Data": encoding classical data into
 * the basis state or into the amplitude vector; angle encoding is rotation
 * gates bound to inputs).
 *   QL_EMBED_NONE       |0...0>.
 *   QL_EMBED_BASIS      qubit q is 1 where inputs[b][first + q] >= 0.5 (a
 *                       direct-product basis state); no gradient.
 *   QL_EMBED_AMPLITUDE  psi_0 = x / |x| for the 2^n real features
 *                       x = inputs[b][first .. first + 2^n - 1] (n <= 30; a
 *                       zero vector gives the zero state: <Z> = 0, no
 *                       gradient). grad_inputs of those features is the VJP
 *                       through the normalisation,
 *                       (2 / |x|) (Re lambda_0 - psi_0 Re<psi_0|lambda_0>),
 *                       with lambda_0 the adjoint state after the sweep. */
enum { QL_EMBED_NONE = 0, QL_EMBED_BASIS = 1, QL_EMBED_AMPLITUDE = 2 };

/* Circuit extras for ql_circuit_create_desc. pauli_p[c][3] = (p_x, p_y, p_z)
 * of the c-th QL_PAULI gate in gate order (each >= 0, sum <= 1); read during
 * the call only. NULL when the circuit has no Pauli channels. */
typedef struct {
    int32_t embedding;      /* QL_EMBED_* */
    int32_t embed_first;    /* first input feature the embedding reads */
    const double* pauli_p;
} ql_circuit_desc;

typedef enum { QL_C64 = 0, QL_C128 = 1 } ql_dtype;

/* Workspace modes. QL_MODE_FWD_BWD_KEEP is ql_forward_backward with the
 * state after every tile pass but the last kept in the workspace: the
 * backward pass over tile pass p+1 then leaves its un-computed state unstored
 * and the one over pass p loads the kept state after pass p instead (one
 * state write fewer per backward pass: 5m - 5 instead of 6m - 6 state
 * transfers for m tile passes), at the cost of m - 2 more states of
 * workspace (m - 1 with an embedding, whose initial state keeps its
 * buffer). ql_forward_backward takes this path whenever its workspace holds
 * ql_workspace_bytes(..., QL_MODE_FWD_BWD_KEEP) bytes; results agree with the
 * other path up to rounding (the backward reads the forward's states rather
 * than re-derived ones). With one tile pass (or the whole-state kernel) there
 * is nothing to keep; with two the kept state takes the place of the psi
 * buffer, the two sizes are equal and the states are always kept. */
enum { QL_MODE_FWD = 0, QL_MODE_FWD_BWD = 1, QL_MODE_FWD_BWD_KEEP = 2 };

enum {
    QL_OK = 0,
    QL_EINVAL = -1,       /* invalid argument (gate, index, pointer, size) */
    QL_ENOMEM = -2,       /* workspace too small, size overflow, host allocation failed */
    QL_EUNSUPPORTED = -3, /* too many qubits for this dtype or option out of range */
    QL_EHIP = -4          /* HIP runtime error (message from hipGetErrorString) */
};

/* Largest qubit count per dtype. */
#define QL_MAX_QUBITS_C64 32
#define QL_MAX_QUBITS_C128 31

/* Optional planning knobs; zero means "library default". They change how the
 * work is split into kernel passes, never the results beyond fp rounding. */
typedef struct {
    int32_t log_regs;           /* amplitudes per thread = 2^log_regs (2..5) */
    int32_t log_threads;        /* threads per workgroup = 2^log_threads (6..9) */
    int32_t low_qubits;         /* qubits 0..low_qubits-1 are in every tile (1..8) */
    int32_t max_gates_per_pass; /* cap on gates per tile pass (>= 1) */
    int32_t force_tiled;        /* kernel choice: 0 library default (register tiles for
                                   n >= 8, a whole-state kernel below), 1 register
                                   tiles, -1 a whole-state kernel whenever it fits
                                   (n <= 12 for QL_C64, n <= 11 for QL_C128). The
                                   whole-state kernels hold a sample in one
                                   wavefront's registers for n <= 8 (in LDS for
                                   forward-only launches of 2048 or more circuits)
                                   and in LDS above */
    int32_t wg_per_sample;      /* workgroups per sample in a tile pass */
    int32_t rz_groups;          /* 0: RZs on the register bits of one tile layout that
                                   commute into one place (at least three, on distinct
                                   bits) run as one per-register phase op, and an RZ
                                   that commutes back to an RY on its bit runs in one
                                   op with it; -1: every RZ runs on its own */
    int32_t pass_search;        /* how the tiles of the passes are chosen. 1: one pass
                                   at a time, the candidate whose pass plus a greedy
                                   completion of the rest is cheapest under a
                                   memory/arithmetic cost model (no nearly empty
                                   passes at the end of long CNOT chains); -1: one
                                   pass at a time, the candidate that runs the most
                                   gates; 0 (default): a beam search over whole pass
                                   sequences, taken when it needs fewer passes than
                                   1, else 1 */
    int32_t product_prefix;     /* the one-qubit gates a qubit meets before any
                                   two-qubit gate or Pauli channel touches it (the
                                   product-state prefix of the circuit) need not
                                   run as tile ops: the first pass can start from
                                   the product state they make (per-sample
                                   factors, fp64), and their gradients come from
                                   each qubit's environment in lambda at the end of
                                   the backward sweep (tile plans without an
                                   embedding). 0 (default): so when the other gates
                                   then plan into fewer passes, or as many with no
                                   more layout changes; 1: always; -1: never */
    int32_t cz_groups;          /* 0: two or more CZs of one tile layout that commute
                                   into one place (each with at least one operand
                                   outside the registers, or on two register bits)
                                   run as one sign op; -1: every CZ runs on its own */
} ql_options;

typedef struct ql_circuit ql_circuit; /* opaque */

/* Validate the gate list and build the pass plans for both dtypes.
 * n_qubits in [1, 32]; gates[n_gates] as above; n_inputs features per sample
 * and n_weights trainable weights index the angle sources. The gate list is
 * copied. Returns QL_EINVAL for a bad qubit, q0 == q1, a wrong source for the
 * kind, an index out of range or a NULL pointer. */
int ql_circuit_create(int32_t n_qubits, const ql_gate* gates, int32_t n_gates,
                      int32_t n_inputs, int32_t n_weights, ql_circuit** out);

/* Same with planning options (NULL = defaults). */
int ql_circuit_create_ex(int32_t n_qubits, const ql_gate* gates, int32_t n_gates,
                         int32_t n_inputs, int32_t n_weights, const ql_options* opts,
                         ql_circuit** out);

/* Same with an initial-state embedding and Pauli-channel probabilities (desc
 * NULL = no embedding, no channels) and planning options (NULL = defaults).
 * Returns QL_EINVAL also for an embedding whose features do not fit in
 * n_inputs, amplitude embedding above 30 qubits, a QL_PAULI gate without
 * probabilities, or probabilities < 0 or summing above 1. Every entry point
 * honours the embedding and the channels. */
int ql_circuit_create_desc(int32_t n_qubits, const ql_gate* gates, int32_t n_gates,
                           int32_t n_inputs, int32_t n_weights, const ql_circuit_desc* desc,
                           const ql_options* opts, ql_circuit** out);

/* Free a handle (NULL is a no-op). Waits only for the queued table uploads
 * of calls made with it (an event per stream that made any), not for other
 * work on the device. The handle must not be used afterwards. */
void ql_circuit_destroy(ql_circuit* c);

/* Bytes of device workspace a call with this dtype, batch and mode
 * (QL_MODE_*) needs. */
int ql_workspace_bytes(const ql_circuit* c, ql_dtype dtype, int64_t batch, int mode,
                       size_t* out);

/* Forward: inputs[batch][n_inputs], weights[n_weights] -> expz[batch][n_qubits].
 * inputs may be NULL when n_inputs == 0, weights when n_weights == 0. */
int ql_forward(const ql_circuit* c, ql_dtype dtype, int64_t batch,
               const void* inputs, const void* weights, void* expz,
               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Forward + adjoint VJP. grad_out[batch][n_qubits] is the upstream gradient;
 * grad_inputs[batch][n_inputs] and grad_weights[n_weights] may each be NULL
 * (not computed). expz is written as in ql_forward. */
int ql_forward_backward(const ql_circuit* c, ql_dtype dtype, int64_t batch,
                        const void* inputs, const void* weights, const void* grad_out,
                        void* expz, void* grad_inputs, void* grad_weights,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Allocation-free forward + backward, for callers that cannot allocate
 * device memory or pass a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation).
 *
 * Same arguments, results and errors as ql_forward_backward without the
 * workspace: the call runs in a static device buffer of
 * QL_STATIC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends, and returns QL_ENOMEM (before launching anything)
 * when the circuit, dtype and batch need more than that
 * (ql_workspace_bytes(..., QL_MODE_FWD_BWD) tells). It calls no device or
 * host allocator: the plan tables are copied from the handle's own host copy.
 * The caller still provides inputs and outputs. All calls on one GPU share
 * that GPU's buffer: calls that overlap in time on one GPU (other streams,
 * other threads) race and give wrong results; serialise them. Nothing in the
 * buffer needs to start at zero, so its contents from an earlier call do not
 * matter. */
#define QL_STATIC_SCRATCH_BYTES (64u << 20)
int ql_forward_backward_static(const ql_circuit* c, ql_dtype dtype, int64_t batch,
                               const void* inputs, const void* weights, const void* grad_out,
                               void* expz, void* grad_inputs, void* grad_weights,
                               hipStream_t stream);
/* ---- parameter-shift gradients -------------------------------------------
 *
 * The same VJP as ql_forward_backward, computed with the two-term
 * parameter-shift rule instead of the adjoint sweep. The paper's hybrid example
 * (appendix, class Hybrid) differentiates its quantum node this way, by
 * re-running the circuit with the angle shifted by +pi/2 and -pi/2; for
 * exp(-i t P / 2) gates d<Z_i>/dt = (<Z_i>(t + pi/2) - <Z_i>(t - pi/2)) / 2 is
 * exact (the paper's own expression omits the 1/2). Every rotation occurrence
 * s of every sample b gives two shifted circuits; together with the unshifted
 * one these are B * (2S + 1) circuits for S rotation gates, run as extra
 * samples of batched forward passes in chunks of at most max_chunk circuits
 * (0 = all at once). Arguments, outputs, layout and errors are those of
 * ql_forward_backward; grad_out is required. The workspace must hold
 * ql_param_shift_workspace_bytes(c, dtype, batch, max_chunk) bytes; it grows
 * with the chunk (one state per circuit of a chunk) and with B * (2S + 1)
 * fp64 values. Results are deterministic.
 *
 * A controlled rotation CR(t) equals R(t/2) E R(-t/2) E (E = CNOT for CRY and
 * CRZ, CZ for CRX); its two half-angle rotations are shifted separately and
 * their differences combined with factors +-1/2, which is exact (it equals
 * the four-term rule for the controlled generator). Pauli channels are not
 * shifted. With QL_EMBED_AMPLITUDE, grad_inputs must be NULL
 * (QL_EUNSUPPORTED otherwise): the shift rule gives no gradient for
 * amplitudes. */
int ql_param_shift_workspace_bytes(const ql_circuit* c, ql_dtype dtype, int64_t batch,
                                   int64_t max_chunk, size_t* out);
int ql_param_shift(const ql_circuit* c, ql_dtype dtype, int64_t batch, const void* inputs,
                   const void* weights, const void* grad_out, void* expz, void* grad_inputs,
                   void* grad_weights, int64_t max_chunk, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/* ---- final states and shot sampling --------------------------------------
 *
 * The paper's quantum node measures its circuit with a finite number of shots
 * (Sec. "Quantum Node"; the appendix examples measure 100 shots and turn the
 * counts into probabilities). These calls expose that measurement: ql_state
 * writes the final state of every sample, and ql_sample draws shots from
 * states with caller-supplied uniforms.
 *
 * ql_state: same inputs as ql_forward; psi[batch][2^n_qubits] receives the
 * final state (interleaved complex: float2 for QL_C64, double2 for QL_C128),
 * a caller-owned device buffer that also serves as the working state (the
 * workspace then holds no state). Workspace from ql_state_workspace_bytes. */
int ql_state_workspace_bytes(const ql_circuit* c, ql_dtype dtype, int64_t batch, size_t* out);
int ql_state(const ql_circuit* c, ql_dtype dtype, int64_t batch, const void* inputs,
             const void* weights, void* psi, void* workspace, size_t workspace_bytes,
             hipStream_t stream);

/* ql_sample: psi[batch][2^n_qubits] (device, the layout of ql_state) and
 * uniforms[batch][shots] (device, fp64 in [0, 1)); samples[batch][shots]
 * (device, int64) receives, for shot s of sample b, the smallest basis index j
 * whose running sum of |psi_i|^2 (i <= j, in index order) exceeds
 * uniforms[b][s] times the state's total |psi|^2 -- the inverse-CDF draw, so
 * the index's bits are the measured qubits (qubit q = bit q) and no
 * zero-probability index is returned. The sums run in fp64 in a fixed
 * (blocked) order; when a uniform falls within rounding of a CDF boundary the
 * neighbouring index may be returned. zhat[batch][n_qubits] (device, fp32 for
 * QL_C64, fp64 for QL_C128; may be NULL) receives the shot estimate of <Z_q>:
 * (shots with bit q = 0 minus shots with bit q = 1) / shots. The states need
 * not be normalised. shots = 0 writes nothing. Workspace:
 * ql_sample_workspace_bytes(n_qubits, batch) bytes (per block of up to 4096
 * amplitudes, the prefix of block totals and the block's 64 chunk sums:
 * 65 fp64). n_qubits in [1, 32] (QL_C128: [1, 31]). */
int ql_sample_workspace_bytes(int32_t n_qubits, int64_t batch, size_t* out);
int ql_sample(ql_dtype dtype, int32_t n_qubits, int64_t batch, const void* psi, int64_t shots,
              const double* uniforms, int64_t* samples, void* zhat, void* workspace,
              size_t workspace_bytes, hipStream_t stream);

/* Message of the last failing call on this thread ("" if none). */
const char* ql_last_error(void);

/* ---- introspection (host only, no GPU needed) ---------------------------- */

typedef struct {
    int32_t kernel;        /* 0 = whole state in LDS (one workgroup per sample), 1 = tile passes */
    int32_t n_passes;      /* forward tile passes (1 for the whole-state kernel) */
    int32_t tile_qubits;   /* qubits per tile (log2 amplitudes per workgroup tile) */
    int32_t log_regs;      /* amplitudes per thread = 2^log_regs */
    int32_t log_threads;   /* threads per workgroup = 2^log_threads */
    int32_t low_qubits;    /* contiguous low qubits in every tile */
    int32_t n_transposes;  /* LDS layout changes summed over the forward passes */
    int32_t n_param_gates; /* rotation occurrences bound to inputs or weights (S of the
                              parameter-shift count; a controlled rotation counts 2) */
    int32_t n_lane_swaps;  /* in-register layout changes (register bit <-> lane bit) summed
                              over the forward passes */
    int32_t n_rz_groups;   /* RZ groups (several RZs run as one phase op), all passes */
    int32_t n_ryz_pairs;   /* RZs run together with their bit's RY in one op, all passes */
    int32_t n_prefix_gates; /* gates of the product-state prefix (the first pass's initial
                               state; see ql_options.product_prefix) */
    int32_t n_cz_groups;   /* CZ groups (several CZs run as one sign op), all passes */
} ql_plan_info;

int ql_plan_info_get(const ql_circuit* c, ql_dtype dtype, ql_plan_info* out);

/* Forward schedule: pass_of_gate[n_gates] receives the pass that applies each
 * gate, order[n_gates] the gate indices in execution order (pass by pass).
 * Gates of the product-state prefix belong to pass 0 and come first, in gate
 * order. A controlled rotation or Pauli channel runs as several gates; it is
 * reported at the pass and position of the last one (a channel with all
 * probabilities 0 applies nothing: pass -1, listed first). */
int ql_plan_schedule(const ql_circuit* c, ql_dtype dtype, int32_t* pass_of_gate,
                     int32_t* order);

/* Algorithmic HBM bytes of the state passes of one call in a mode (QL_MODE_*:
 * reads + writes of psi and lambda by the tile kernel; 0 for the whole-state
 * kernel). */
int ql_plan_state_bytes(const ql_circuit* c, ql_dtype dtype, int64_t batch, int mode,
                        double* out);

/* ---- timing (for benchmarks) --------------------------------------------- */

/* Kernel classes: 0 tile passes, 1 whole-state kernel, 2 angle binding and
 * embedding, 3 reductions. enable = 0 turns timing off; otherwise bit c of
 * enable selects class c (15: all). Every launch of a selected class is then
 * bracketed by HIP events on the call's stream (each pair costs host time,
 * which shows on launch-bound workloads: time only the classes needed).
 * ql_timing_read synchronises on the last event and returns the summed
 * milliseconds per class in ms[0..3] and the launch counts in
 * launches[0..3]. Reading resets them. Not thread-safe: one timed call in
 * flight per handle. */
int ql_timing_enable(ql_circuit* c, int enable);
int ql_timing_read(ql_circuit* c, double ms[4], int32_t launches[4]);

#ifdef __cplusplus
}
#endif

#endif /* QLAYER_H */
