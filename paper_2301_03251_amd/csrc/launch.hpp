// launch.hpp -- host-side launchers of the HIP kernels (kernels.hip, tile.hip).
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "plan.hpp"

namespace qlayer {

// Source of a slot; one row per slot. Rotation slots: angle = scale * the
// bound input or weight. Pauli-channel slots (src S_PAULI): the uniform input
// feature `index` selects X if u < c1, Y if u < c2, Z if u < c3, else none.
struct SlotSrc {
    int32_t src, index;
    double scale;
    double c1, c2, c3;
};

// Whole-state (one workgroup per sample, state in LDS) gate entry.
struct DevGate {
    int32_t kind, q0, q1, slot;
};

struct BindArgs {
    const void* inputs;   // [B][F] Real
    const void* weights;  // [P] Real
    const SlotSrc* slots; // [n_slots]
    void* coef;           // [B][n_slots] complex (cos, sin) of theta/2; a Pauli slot: (which, 0)
    int64_t B;
    int32_t n_slots, F;
    int64_t v0;           // parameter-shift chunks: first virtual circuit
    int32_t vper;         // circuits per sample (2 * n_slots + 1), 0 = plain batch
};

// Per-sample records of the tile ops (handler id, argument, two shear
// coefficients of the rotation angle); ops at index >= bwd_first belong to
// backward ranges and get the inverse rotation.
struct BindTileArgs {
    const void* inputs;    // [B][F] Real
    const void* weights;   // [P] Real
    const SlotSrc* slots;  // [n_slots]
    const DevOp* ops;      // [n_ops]
    void* opc;             // [B][n_ops + 1] records
    const DevDiag* diags;  // [n_diags] RZ groups
    void* dzc;             // [B][n_diags][DZ_REGS] complex: (cos, sin) of each register's phase
    int32_t n_diags;
    const DevFuse* fuses;  // [n_fuses] RZs of RY-RZ pair ops
    void* fzc;             // [B][n_fuses] (a, b) shear coefficients of each pair's RZ (forward)
    int32_t n_fuses;
    int64_t B;
    int32_t n_ops, bwd_first, F;
    int64_t v0;            // parameter-shift chunks: first virtual circuit
    int32_t vper;          // circuits per sample (2 * n_slots + 1), 0 = plain batch
};

// Parameter shift: per shifted circuit v of a chunk, d[v] = sum_i grad_out[b][i]
// * ev[v - v0][i] in fp64 (b = v / vper); the unshifted circuit (v % vper == 0)
// also writes expz[b].
struct ShiftDotArgs {
    const void* ev;        // [count][n] Real: <Z> of the chunk's circuits
    const void* grad_out;  // [B][n] Real
    void* expz;            // [B][n] Real
    double* dv;            // [B * vper]
    int64_t v0, count;
    int32_t vper, n;
};

// grad of rotation slot s of sample b = (d[b, 2s+1] - d[b, 2s+2]) / 2, summed
// over each input's / weight's slots (and over the batch for weights).
struct ShiftGradArgs {
    const double* dv;      // [B * vper]
    void* grad_inputs;     // [B][F] Real or null
    void* grad_weights;    // [P] Real or null
    const int32_t* x_ptr;
    const int32_t* x_slot;
    const int32_t* w_ptr;
    const int32_t* w_slot;
    const SlotSrc* slots;  // scales of the rotation slots
    int64_t B;
    int32_t vper, F, P;
};

struct WholeArgs {
    const DevGate* gates;
    int32_t n_gates, n, n_slots;
    int32_t bwd;          // 1: run the adjoint sweep
    int64_t B;
    const void* coef;     // [B][n_slots]: from k_bind (LDS kernel), unused by the wavefront kernel
    // the angle sources, which the one-wavefront kernel binds itself (as k_bind does)
    const SlotSrc* slots; // [n_slots]
    const void* inputs;   // [B][F] Real
    const void* weights;  // [P] Real
    int32_t F;
    int32_t vper;         // parameter-shift chunks: circuits per sample, 0 = plain batch
    int64_t v0;           // parameter-shift chunks: first virtual circuit
    const void* grad_out; // [B][n] Real
    double* zpart;        // [B][n]           (one workgroup per sample)
    double* gpart;        // [n_slots][B]
    void* psi_out;        // [B][2^n] complex: the final state, or null
    const void* psi_in;   // [B][2^n] complex: the initial state, or null for |0...0>
    void* lam_out;        // [B][2^n] complex: lambda after the backward sweep, or null
};

// Initial-state embeddings: circuit i of a call (sample i, or sample
// (v0 + i) / vper of a parameter-shift chunk) starts from the basis state of
// features first..first+n-1 (>= 0.5 is a 1) or from x / |x| over the 2^n
// features from `first` on.
struct EmbedArgs {
    const void* inputs;   // [B][F] Real
    void* psi;            // [count][2^n] complex
    double* norm;         // [count]: |x| (amplitude embedding)
    int64_t count;        // circuits
    int64_t v0;
    int32_t vper;         // 0: circuit i is sample i
    int32_t kind, first, F, n;
};

// Amplitude-embedding VJP: grad_inputs[b][first + j] += (2 / |x|) (Re lam_j -
// psi0_j L_b) with L_b = sum_j psi0_j Re lam_j (dot: [B] fp64 scratch).
struct EmbedGradArgs {
    const void* inputs;   // [B][F] Real
    const void* lam;      // [B][2^n] complex: lambda_0
    const double* norm;   // [B]
    double* dot;          // [B]
    void* grad_inputs;    // [B][F] Real
    int64_t B;
    int32_t first, F, n;
};

// Shot sampling from states psi[B][2^n]: blocks of 2^bb amplitudes, each
// split into 64 lane chunks.
struct SampleArgs {
    const void* psi;        // [B][2^n] complex
    const double* uniforms; // [B][shots] in [0, 1)
    int64_t* samples;       // [B][shots]
    void* zhat;             // [B][n] Real or null: <Z_q> estimated from the shots
    double* bsum;           // [B][nblk]: block sums, then their inclusive prefix
    double* csum;           // [B][nblk][64]: each block's 64 lane-chunk sums
    int64_t B, shots, nblk;
    int32_t n, bb;
};

// Registers of an RZ group's phase table (one entry per register index).
constexpr int DZ_REGS = 1 << MAX_DZ_BITS;

struct TileArgs {
    const void* psi;           // [B][2^n] complex: loaded state
    void* psi_out;             // [B][2^n] complex: stored state (psi itself, or another buffer)
    void* lam;                 // [B][2^n] complex
    const DevPass* pass;
    const DevPhase* phases;
    const DevOp* ops;
    const int32_t* gslots;     // pass-local gradient index -> rotation slot
    const void* opc;           // [B][n_ops + 1] per-sample op records
    const void* dzc;           // [B][n_diags][DZ_REGS] RZ-group phase tables
    int32_t n_diags;
    const void* fzc;           // [B][n_fuses] RZ coefficients of the RY-RZ pair ops
    int32_t n_fuses;
    const void* grad_out;      // [B][n] Real
    double* zpart;             // [B][n_wg][n]
    double* gpart;             // [n_slots][B][n_wg]
    int64_t B;
    int64_t tiles;             // tiles per sample = 2^(n-k)
    int32_t n, n_ops, n_wg, flags;
    int32_t n_gslots;          // gradient accumulators of this pass
    const double* phi;         // [B][n][2] complex (double2): product-prefix factors (PF_PRODUCT)
    const DevCzg* czg;         // CZ groups (H_CZG ops)
    const uint32_t* pthr;      // [n_phases][PTHR_WORDS] thread layouts of every phase
};

// Product-state prefix. Binding: phi[c][q] = the state the prefix gates of
// qubit q make from |0> (fp64), for every circuit c of the call (parameter-
// shift chunks as in BindArgs). Environment: from lambda at the end of the
// backward sweep, each workgroup's share of r_q(v) = sum over amplitudes i
// with bit q = v of lambda(i) conj(prod_{q' != q} phi_q'(bit q' of i)), as
// (re, im of v = 0, re, im of v = 1) per qubit. Gradients: r_q summed over the
// workgroups and, for prefix gate j of qubit q, d = Im <g_j| P_j |f_j> with
// f_j the factor after gate j and g_j r_q un-applied through the gates after
// j; written to gpart[slot][b][0] (zeros in the other workgroup columns).
struct PrefixArgs {
    const void* inputs;        // [B][F] Real
    const void* weights;       // [P] Real
    const SlotSrc* slots;
    const int32_t* pre_ptr;    // [n + 1]
    const DevPrefix* pre_ops;
    double* phi;               // [count][n][2] complex
    const void* lam;           // [B][2^n] complex: lambda at the end of the backward sweep
    double* envpart;           // [B][env_wg][n][4]
    double* gpart;             // [n_slots][B][n_wg]
    int64_t B;                 // circuits
    int64_t v0;
    int32_t vper;
    int32_t n, F, n_wg;
    int32_t env_wg;            // workgroups per sample of the environment kernel
};
// Workgroups per sample of the environment kernel for n qubits and batch B.
int env_workgroups(int dtype, int n, int64_t B);
// LDS words per (gradient accumulator, wavefront) of the tile kernel
constexpr int TILE_GRAD_WORDS = 2;

struct ReduceArgs {
    const double* zpart;   // [B][n_wg][n]
    const double* gpart;   // [n_slots][B][n_wg]
    void* expz;            // [B][n] Real
    void* grad_inputs;     // [B][F] Real or null
    void* grad_weights;    // [P] Real or null
    const int32_t* x_ptr;  // [F+1] CSR: rotation slots bound to input f
    const int32_t* x_slot;
    const int32_t* w_ptr;  // [P+1] CSR: rotation slots bound to weight p
    const int32_t* w_slot;
    const SlotSrc* slots;  // scales of the rotation slots
    int64_t B;
    int32_t n, n_wg, F, P, n_slots;
    int32_t grads;         // 1: reduce gradients too
};

// Static LDS of a tile kernel: the exchange buffer for a whole tile of
// MAXT threads x 2^LOG_R amplitudes.
template <typename Real, int LOG_R, int MAXT>
constexpr size_t tile_lds_bytes() {
    return (size_t)MAXT * ((size_t)1 << LOG_R) * 2 * sizeof(Real);
}
size_t tile_static_lds(int dtype, int log_r, int threads);

// dtype: 0 = complex64 / fp32, 1 = complex128 / fp64. Return hipError_t.
hipError_t launch_bind(int dtype, const BindArgs& a, hipStream_t s);
hipError_t launch_bind_tile(int dtype, const BindTileArgs& a, hipStream_t s);
hipError_t launch_whole(int dtype, const WholeArgs& a, int threads, size_t lds, hipStream_t s);
// Whether launch_whole runs the one-wavefront kernel (which binds the angles
// itself, so no k_bind launch is needed) for this call.
bool whole_uses_wave(int n, bool bwd, int64_t B);
hipError_t launch_tile(int dtype, int log_r, bool bwd, const TileArgs& a, int threads, size_t lds,
                       hipStream_t s);
hipError_t launch_reduce(int dtype, const ReduceArgs& a, hipStream_t s);
hipError_t launch_shift_dot(int dtype, const ShiftDotArgs& a, hipStream_t s);
hipError_t launch_sample(int dtype, const SampleArgs& a, hipStream_t s);
// Undo the per-sample global phase the tile kernel leaves on final states
// (phase: [2B] fp64 scratch: the inverse phase factor per sample).
hipError_t launch_state_phase(int dtype, const BindTileArgs& a, double* phase, void* psi, int n,
                              hipStream_t s);
hipError_t launch_embed(int dtype, const EmbedArgs& a, hipStream_t s);
hipError_t launch_embed_grad(int dtype, const EmbedGradArgs& a, hipStream_t s);
hipError_t launch_shift_grad(int dtype, const ShiftGradArgs& a, hipStream_t s);
hipError_t launch_bind_prefix(int dtype, const PrefixArgs& a, hipStream_t s);
hipError_t launch_env(int dtype, const PrefixArgs& a, hipStream_t s);
hipError_t launch_env_grad(int dtype, const PrefixArgs& a, hipStream_t s);

// Raise the dynamic-LDS limit of every kernel on the current device.
hipError_t configure_kernels(size_t max_lds);
// The same for the tile kernels only (tile.hip).
hipError_t configure_tile_kernels(size_t max_lds);

}  // namespace qlayer
