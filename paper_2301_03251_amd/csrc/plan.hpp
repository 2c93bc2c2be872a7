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

// Gate kinds the planner and kernels run. The public kinds 6..9 (controlled
// rotations, Pauli-channel trajectories) are rewritten into these at intake;
// K_PAULI is one channel trajectory on q0 whose Pauli (or none) each sample
// draws from its uniform (slot of kind S_PAULI).
enum GateKind { K_H = 0, K_RX = 1, K_RY = 2, K_RZ = 3, K_CNOT = 4, K_CZ = 5, K_PAULI = 16 };
enum PublicKind { P_CRX = 6, P_CRY = 7, P_CRZ = 8, P_PAULI = 9 };
// Sources of slots: rotation angles from inputs or weights; S_PAULI marks a
// channel slot (the Pauli a uniform input feature selects).
enum Src { S_NONE = 0, S_INPUT = 1, S_WEIGHT = 2, S_PAULI = 3 };
enum Embed { E_NONE = 0, E_BASIS = 1, E_AMPLITUDE = 2 };

// One rotation occurrence or Pauli channel after intake. Input and weight
// slots have angle scale * value; a Pauli-channel slot selects X if its
// uniform u (input feature `index`) is < c1, Y if < c2, Z if < c3, else none.
struct Slot {
    int32_t src, index;
    double scale;
    double c1, c2, c3;   // Pauli slots: cumulative probabilities
};

struct Gate {
    int32_t kind, q0, q1, src, index;
    int32_t slot;  // rotation slot (coefficient + gradient), -1 otherwise
    int32_t user;  // index of the gate as given that this gate came from
};

// Operand location relative to the current tile phase.
enum LocType : uint8_t { LOC_REG = 0, LOC_THR = 1, LOC_FIX = 2 };

// Handler ids of tile ops: a dense enumeration so the kernels dispatch every op
// with one switch onto a handler whose register indices are compile-time
// constants.
enum HandlerId : uint32_t {
    H_G1 = 0,          // + kind * 5 + J: H, RX, RY or RZ on register bit J; arg = gradient slot
    H_RZU = 20,        // RZ on a thread bit or fixed qubit; arg = loc | gslot << 16
    H_CNOT_RR = 21,    // + J * 5 + m: target register bit J, control register bit m
    H_CNOT_T = 46,     // + J: control is a thread bit (arg = tile bit)
    H_CNOT_F = 51,     // + J: control is a fixed qubit (arg = qubit)
    H_CZ_RR = 56,      // + a * 5 + b: both register bits
    H_CZ_RX = 81,      // + a: register bit a, other operand in arg (loc)
    H_CZ_XX = 86,      // both operands thread/fixed bits: arg = loc_a | loc_b << 16
    H_TRANSPOSE = 87,  // arg = phase index
    H_RZN = 88,        // + J: RZ on register bit J whose phase on bit 1 is negated (set per sample
                       //      by the binding kernel in place of H_G1 + 15 + J)
    H_LSWAP = 93,      // + m * 6 + b: exchange register bit m with lane bit b (4 or 5) by
                       //      permlane swaps; arg = lswap_arg(new phase, tile bit lane b
                       //      leaves, tile bit it takes)
    H_PX = 123,        // + P * 5 + J: Pauli X (P = 0), Y (1) or Z (2) on register bit J; a
                       //      channel op is planned as H_PX + J and set per sample by the
                       //      binding kernel to the Pauli its uniform selects, or to H_NOP
    H_DZ = 138,        // RZ group: the RZs of up to MAX_DZ_BITS register bits in one diagonal
                       //      op (a per-register phase); arg = group index (DevDiag)
    H_RYZ = 139,       // + J: RY then RZ on register bit J in one op; arg = RY gradient slot |
                       //      RZ gradient slot << 8 | pair index (DevFuse) << 16
    H_RYZN = 144,      // + J: the same with the RZ's phase negated (chosen per sample by the
                       //      binding kernel, as H_RZN for a single RZ)
    H_NOP = 149,
    H_END = 150,
    H_CZG = 151,       // CZ group: the CZs of one layout in one sign op; arg = group index (DevCzg)
};
// The RZ of an RY-RZ pair op (H_RYZ): its rotation slot and gradient slot.
struct DevFuse {
    int32_t slot;
    uint32_t gslot;
};
// Register bits an RZ group can span (its gradient slots travel in the op
// record's two coefficient words, 16 bits each).
constexpr int MAX_DZ_BITS = 4;
// An RZ group is formed from at least this many RZs: below it the separate
// ops cost less than a phase on every register.
constexpr int MIN_DZ_SIZE = 3;

// Members of an RZ group, by register bit J: the rotation slot and the
// gradient slot of the RZ on bit J (-1 / NO_GSLOT: no RZ on that bit).
struct DevDiag {
    int32_t slot[MAX_DZ_BITS];
    uint32_t gslot[MAX_DZ_BITS];
};
static_assert(sizeof(DevDiag) == 32, "DevDiag layout");
// A CZ group: CZs of one tile layout that commute into one place, applied as
// one sign pattern. An amplitude is negated when an odd number of the pairs
// have both operand bits set. Register operands are register bits of the
// layout; the other operands are thread bits (tile bits the lanes hold) or
// fixed qubits (uniform per tile).
constexpr int CZG_REG_BITS = 5;    // register bits of the largest register tile
constexpr int MAX_CZG_PAIRS = 16;  // pairs with no register operand per group
struct DevCzg {
    uint32_t reg_mask;             // registers negated by the pairs of two register bits
    uint32_t n_tt;                 // pairs of two thread bits: pair[0 .. n_tt)
    uint32_t n_pairs;              // then thread-fixed and fixed-fixed pairs up to n_pairs
    uint32_t thr[CZG_REG_BITS];    // per register bit: tile-bit mask of its thread-bit partners
    uint32_t fix[CZG_REG_BITS];    // per register bit: qubit mask of its fixed-qubit partners
    uint32_t pair[MAX_CZG_PAIRS];  // thread-thread: tile bits a | b << 8; others: loc words a | b << 16
    uint32_t pad[3];
};
static_assert(sizeof(DevCzg) == 128, "DevCzg layout");
// Argument of a lane swap: the new phase (< 2^20) and the tile bits x (leaving
// the lane bit for the registers) and y (taking its place).
constexpr uint32_t lswap_arg(uint32_t phase, uint32_t x, uint32_t y) {
    return phase | x << 20 | y << 25;
}
// A loc in an op argument: tile bit or qubit in bits 0..7, LocType in bits 8..9.
constexpr uint32_t loc_word(uint32_t type, uint32_t pos) { return pos | (type << 8); }
constexpr uint32_t NO_GSLOT = 0xffffu;
// Flag in the argument of a backward layout change (H_TRANSPOSE, H_LSWAP):
// refresh the thread's Im<lambda|psi> sum after it, because an RZ-type
// gradient term uses that sum before the next layout change.
constexpr uint32_t ARG_IVAL = 1u << 30;

// Static op of a tile pass (the binding kernel turns it into a per-sample record).
struct DevOp {
    uint32_t h;      // handler id
    uint32_t arg;    // handler argument (H_G1: gradient slot or NO_GSLOT)
    int32_t slot;    // rotation slot (angle source), -1 none
    uint32_t kind;   // gate kind (K_*), or K_H for non-gates
};
static_assert(sizeof(DevOp) == 16, "DevOp layout");

// Gradient accumulators per pass (one per rotation in the pass).
constexpr int MAX_GSLOTS = 256;

constexpr int MAX_LOG_R = 5;
constexpr int MAX_R = 1 << MAX_LOG_R;
constexpr int MAX_TILE_BITS = 16;

constexpr int MAX_THREAD_BITS = 12;

// Register layout of one phase: register bit m of a thread's amplitude index
// is tile bit reg_bit[m]; thread-index bit b is tile bit thr_bit[b] (bits 0-5
// are lane bits, the rest wavefront bits). Every per-register and
// per-thread-bit offset the kernel needs is precomputed here, so a layout
// change costs one XOR per access.
//
// LDS: the amplitude with tile index t sits in slot lds_slot(t) (a GF(2)-linear
// bank-spreading permutation), so the byte offset of (thread, register i) is
// XOR(thr_slot[b] for set bits b of the thread index) ^ reg_slot[i].
struct DevPhase {
    uint32_t thr_mask;                   // tile bits held by the thread index
    uint32_t reg_bit[MAX_LOG_R];         // register bit m -> tile bit
    uint32_t reg_tmask[MAX_LOG_R];       // 1 << reg_bit[m]
    uint32_t reg_qmask[MAX_LOG_R];       // 1 << (qubit of tile bit reg_bit[m])
    uint32_t thr_bit[MAX_THREAD_BITS];   // thread-index bit b -> tile bit
    uint32_t thr_slot[MAX_THREAD_BITS];  // LDS byte offset of thread-index bit b
    uint32_t reg_slot[MAX_R];            // LDS byte offset of register i's tile bits
    uint32_t reg_qoff[MAX_R];            // amplitude-index offset of register i's tile bits
};

// Thread layouts of a phase as tables: PTHR_WORDS words per phase, 64 for
// the lane bits (indexed by lane) and 8 for the wavefront bits (indexed by
// wavefront); each word holds the tile bits (low PTHR_TB_BITS bits: k <= 14)
// and the LDS byte offset (above) that those thread-index bits contribute.
constexpr int PTHR_WORDS = 72;
constexpr int PTHR_TB_BITS = 14;
// Bank-spreading permutation of LDS slots: folds the upper nibbles of the tile
// index into the lowest one. Linear over GF(2), an involution on each aligned
// block of 2^16 slots.
constexpr uint32_t lds_slot(uint32_t t) { return t ^ (((t >> 4) ^ (t >> 8) ^ (t >> 12)) & 15u); }

enum PassFlags : int32_t {
    PF_INIT = 1,        // start from |0..0> instead of loading psi
    PF_LOAD_LAM = 2,    // load lambda (separate backward pass)
    PF_FWD = 4,         // run the forward ops
    PF_ZPART = 8,       // accumulate <Z_q> partials after the forward ops
    PF_SEED = 16,       // lambda = (sum_q g_q Z_q) psi
    PF_BWD = 32,        // run the backward ops (needs lambda)
    PF_STORE_PSI = 64,
    PF_STORE_LAM = 128,
    PF_PRODUCT = 256,   // start from the product state of the per-sample prefix factors
};

// A gate of a qubit's prefix (its one-qubit gates before any two-qubit gate or
// Pauli channel touches it): kind K_H/K_RX/K_RY/K_RZ and rotation slot (-1 for H).
struct DevPrefix {
    int32_t kind, slot;
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
    int32_t index;           // pass index in the plan
    int32_t tile_qubit[MAX_TILE_BITS];  // tile bit -> qubit
    int32_t fixed_qubit[32];            // ascending qubits outside the tile
    int32_t pad[3];
};

struct Options {
    int log_regs = 0, log_threads = 0, low_qubits = 0, max_gates_per_pass = 0;
    int force_tiled = 0, wg_per_sample = 0;
    int rz_groups = 0;  // 0: RZs on register bits are grouped into H_DZ ops or joined to their
                        // bit's RY (H_RYZ); -1: every RZ runs on its own
    int product_prefix = 0;  // each qubit's leading one-qubit gates form the initial product state
                             // (tile plans without an embedding): 0 when the rest plans no worse,
                             // 1 always, -1 never (they run as ops)
    int cz_groups = 0;  // 0: CZs of one layout that commute into one place run as one H_CZG
                        // op (two or more); -1: every CZ runs on its own
    int pass_search = 0;  // 0: a beam search over pass sequences when it needs fewer passes than
                          // the look-ahead, else the look-ahead; 1: the look-ahead (each
                          // pass's tile priced by its pass plus a greedy completion); -1: the
                          // widest pass each time
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
    int n_transposes = 0;             // layout changes through LDS
    int n_lane_swaps = 0;             // layout changes inside the registers
};

struct Plan {
    bool whole_state = false;  // single-kernel path (state in LDS)
    int n = 0, k = 0, log_r = 0, log_t = 0, low = 0;
    std::vector<PassPlan> passes;
    std::vector<DevPhase> phases;
    std::vector<DevDiag> diags;  // RZ groups (H_DZ ops), all passes
    std::vector<DevFuse> fuses;  // RZs of RY-RZ pair ops (H_RYZ), all passes
    std::vector<DevCzg> czgs;    // CZ groups (H_CZG ops), all passes
    int n_slots = 0;           // rotation slots
    // Product prefix (tile plans): the gates of pre_ops[pre_ptr[q] .. pre_ptr[q+1])
    // act on qubit q of |0...0> before anything else touches it, so the first
    // pass starts from the product of the per-qubit states they make, and the
    // passes hold only the other gates. Empty when product is false.
    bool product = false;
    std::vector<int32_t> pre_ptr;   // [n + 1]
    std::vector<DevPrefix> pre_ops;
    std::vector<int> pre_gates;     // the prefix gates, in gate order
};

// Intake extras: the initial-state embedding and the Pauli-channel
// probabilities ([channels][3], in gate order).
struct Extras {
    int embed = E_NONE, embed_first = 0;
    const double* pauli_p = nullptr;
};

struct Circuit {
    int n = 0, n_inputs = 0, n_weights = 0;
    int embed = E_NONE, embed_first = 0;
    std::vector<Gate> gates;     // after intake: kinds H..CZ only
    std::vector<Slot> slots;     // slots: trainable rotations first, then Pauli channels
    int n_param_slots = 0;       // slots bound to inputs or weights
    int n_user_gates = 0;        // gates as given
    Options opts;
    Plan plan[2];                // per dtype (0 = c64, 1 = c128)
};

// Validate and copy gates, rewrite controlled rotations and Pauli channels
// into rotations and CNOT/CZ, assign rotation slots. Returns "" or an error.
std::string build_circuit(int n, const int32_t* gates5, int n_gates, int n_inputs,
                          int n_weights, const Extras& ext, const Options& opts, Circuit& out);

// Largest qubit count for amplitude embedding (2^n features per sample).
constexpr int AMPLITUDE_MAX_QUBITS = 30;

// Build the plan for one dtype. Returns "" or an error message.
std::string build_plan(const Circuit& c, int dtype, Plan& out);

// Largest qubit count that the whole-state kernel handles for a dtype.
int whole_state_max_qubits(int dtype);

}  // namespace qlayer
