// plan.hpp -- circuit validation and the pass planner (host C++, no HIP).
//
// A circuit on n qubits is applied to a batch of state vectors psi[b][2^n].
// When the whole state of a sample fits in one workgroup's LDS the circuit runs
// in a single whole-state kernel. Otherwise the gate list is cut into tile
// passes: a pass picks a set T of k qubits (the low `low` qubits, for coalesced
// HBM access, plus up to k - low others), and every workgroup loads 2^k
// amplitudes that differ only in the bits of T, applies every gate of the pass
// there and writes them back. Gates that act only on T run inside the tile;
// diagonal gates (RZ, CZ) and CNOTs whose target is in T also run when their
// other qubits lie outside T, because those bits are fixed for the whole tile.
//
// Inside a tile, each thread holds 2^r amplitudes in registers that differ in
// r "register bits" of the tile index; the other k - r tile bits select the
// thread. A gate that mixes amplitude pairs (H, RX, RY, CNOT target) needs its
// tile bit among the register bits; a "phase" is one choice of register bits,
// and switching phase is an exchange of the tile through LDS.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace qlayer {

enum GateKind { K_H = 0, K_RX = 1, K_RY = 2, K_RZ = 3, K_CNOT = 4, K_CZ = 5 };
enum Src { S_NONE = 0, S_INPUT = 1, S_WEIGHT = 2 };

struct Gate {
    int32_t kind, q0, q1, src, index;
    int32_t slot;  // rotation slot (coefficient + gradient), -1 otherwise
};

// Operand location relative to the current tile phase.
enum LocType : uint8_t { LOC_REG = 0, LOC_THR = 1, LOC_FIX = 2 };

enum OpCode : uint8_t {
    OP_G1 = 0,         // H / RX / RY / RZ on register bit a
    OP_RZ_U = 1,       // RZ on a thread bit or fixed qubit (one phase per thread)
    OP_CNOT = 2,       // target register bit a, control b (any location)
    OP_CZ = 3,         // a, b any locations
    OP_TRANSPOSE = 4,  // switch to phase `arg`
};

// Device op: 16 bytes, read with scalar loads.
struct DevOp {
    uint8_t code, kind;
    uint8_t a_type, a_pos;   // target / first operand
    uint8_t b_type, b_pos;   // control / second operand
    uint16_t arg;            // TRANSPOSE: phase index (global in the plan)
    int32_t slot;            // rotation slot (coefficient table column), -1 none
    int32_t gslot;           // pass-local gradient accumulator index, -1 none
};
static_assert(sizeof(DevOp) == 16, "DevOp layout");

constexpr int MAX_LOG_R = 5;
constexpr int MAX_R = 1 << MAX_LOG_R;
constexpr int MAX_TILE_BITS = 16;

// Register layout of one phase.
struct DevPhase {
    uint32_t thr_mask;            // tile bits held by the thread index (ascending -> tid bits)
    uint32_t reg_bit[MAX_LOG_R];  // register position m -> tile bit
    uint32_t reg_off[MAX_R];      // tile-index offset of register i
    uint32_t greg_off[MAX_R];     // amplitude offset (in the sample) of register i
};

enum PassFlags : int32_t {
    PF_INIT = 1,        // start from |0..0> instead of loading psi
    PF_LOAD_LAM = 2,    // load lambda (separate backward pass)
    PF_FWD = 4,         // run the forward ops
    PF_ZPART = 8,       // accumulate <Z_q> partials after the forward ops
    PF_SEED = 16,       // lambda = (sum_q g_q Z_q) psi
    PF_BWD = 32,        // run the backward ops (needs lambda)
    PF_STORE_PSI = 64,
    PF_STORE_LAM = 128,
};

struct DevPass {
    int32_t k;               // tile bits
    int32_t log_t;           // threads per workgroup = 2^log_t
    int32_t n_fixed;         // qubits outside the tile
    int32_t n_gslots;        // gradient accumulators used by the backward ops
    int32_t fwd_begin, fwd_end;         // op ranges in the plan's op table
    int32_t bwd_begin, bwd_end;
    int32_t load_phase;      // layout at the start of the forward ops
    int32_t bwd_phase;       // layout at the start of the backward ops
    int32_t gslot_base;      // first entry in the plan's gslot -> rotation-slot table
    int32_t n_exchanges;     // LDS layout changes in the forward ops
    int32_t tile_qubit[MAX_TILE_BITS];  // tile bit -> qubit
    int32_t fixed_qubit[32];            // ascending qubits outside the tile
};

struct Options {
    int log_regs = 0, log_threads = 0, low_qubits = 0, max_gates_per_pass = 0;
    int force_tiled = 0, wg_per_sample = 0;
};

// One forward tile pass as planned (host form).
struct PassPlan {
    std::vector<int> qubits;          // tile qubits, tile bit order (low qubits first)
    std::vector<int> gates;           // gate indices in execution order
    std::vector<DevOp> fwd_ops;       // with TRANSPOSE entries
    std::vector<DevOp> bwd_ops;
    std::vector<int> gslots;          // pass-local gradient accumulator -> rotation slot
    int first_phase = 0;              // phase index at pass start (forward)
    int last_phase = 0;               // phase index at pass end (forward)
    int n_transposes = 0;
};

struct Plan {
    bool whole_state = false;  // single-kernel path (state in LDS)
    int n = 0, k = 0, log_r = 0, log_t = 0, low = 0;
    std::vector<PassPlan> passes;
    std::vector<DevPhase> phases;
    int n_slots = 0;           // rotation slots
};

struct Circuit {
    int n = 0, n_inputs = 0, n_weights = 0;
    std::vector<Gate> gates;
    std::vector<int> slot_gate;  // rotation slot -> gate index
    Options opts;
    Plan plan[2];                // per dtype (0 = c64, 1 = c128)
};

// Validate and copy gates, assign rotation slots. Returns "" or an error.
std::string build_circuit(int n, const int32_t* gates5, int n_gates, int n_inputs,
                          int n_weights, const Options& opts, Circuit& out);

// Build the plan for one dtype. Returns "" or an error message.
std::string build_plan(const Circuit& c, int dtype, Plan& out);

// Largest qubit count that the whole-state kernel handles for a dtype.
int whole_state_max_qubits(int dtype);

}  // namespace qlayer
