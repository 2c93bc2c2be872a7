// plan.cpp -- circuit validation and the tile-pass planner (host C++, no HIP).
#include "plan.hpp"

#include <algorithm>
#include <cstdio>
#include <set>

namespace qlayer {

namespace {

std::string fmt(const char* f, long a = 0, long b = 0, long c = 0) {
    char buf[256];
    std::snprintf(buf, sizeof buf, f, a, b, c);
    return buf;
}

bool is_rotation(int kind) { return kind == K_RX || kind == K_RY || kind == K_RZ; }

// Tile qubit a gate must hold in the tile (-1: none; diagonal gates and CNOT
// controls can be fixed bits of the tile).
int needed_tile_qubit(const Gate& g) {
    switch (g.kind) {
        case K_H: case K_RX: case K_RY: case K_PAULI: return g.q0;
        case K_CNOT: return g.q1;
        default: return -1;
    }
}

int n_qubits_of(const Gate& g) { return (g.kind == K_CNOT || g.kind == K_CZ) ? 2 : 1; }

// Greedy scan of the not-yet-scheduled gates for a candidate tile qubit set.
// `tile` (a bitmask over qubits) may grow up to `cap` qubits when `grow`.
// Returns the executed gate indices in order. A skipped gate blocks its
// qubits, so every executed gate only commutes past skipped gates acting on
// other qubits.
std::vector<int> scan(const std::vector<Gate>& gates, const std::vector<char>& done,
                      uint64_t& tile, int cap, bool grow, int max_gates) {
    std::vector<int> exec;
    uint64_t blocked = 0;
    int count = __builtin_popcountll(tile);
    int rotations = 0;
    for (int i = 0; i < (int)gates.size(); i++) {
        if (done[i]) continue;
        const Gate& g = gates[i];
        uint64_t qs = (1ull << g.q0) | (n_qubits_of(g) == 2 ? (1ull << g.q1) : 0);
        if (qs & blocked) { blocked |= qs; continue; }
        if (max_gates > 0 && (int)exec.size() >= max_gates) { blocked |= qs; continue; }
        if (is_rotation(g.kind) && rotations >= MAX_GSLOTS) { blocked |= qs; continue; }
        int need = needed_tile_qubit(g);
        bool ok = need < 0 || (tile >> need & 1);
        if (!ok && grow && count < cap) {
            tile |= 1ull << need;
            count++;
            ok = true;
        }
        if (ok) {
            exec.push_back(i);
            rotations += is_rotation(g.kind);
        } else {
            blocked |= qs;
        }
    }
    return exec;
}

// Layout: reg_bits[m] is the tile bit of register bit m, thr_bits[b] the tile
// bit of thread-index bit b. `amp` is the size of one amplitude in bytes (LDS
// offsets are in bytes).
DevPhase make_phase(const std::vector<int>& tq, const std::vector<int>& reg_bits,
                    const std::vector<int>& thr_bits, uint32_t amp) {
    DevPhase p{};
    const int r = (int)reg_bits.size();
    for (int m = 0; m < r; m++) {
        p.reg_bit[m] = reg_bits[m];
        p.reg_tmask[m] = 1u << reg_bits[m];
        p.reg_qmask[m] = 1u << tq[reg_bits[m]];
    }
    for (int b = 0; b < (int)thr_bits.size() && b < MAX_THREAD_BITS; b++) {
        const int j = thr_bits[b];
        p.thr_mask |= 1u << j;
        p.thr_bit[b] = (uint32_t)j;
        p.thr_slot[b] = lds_slot(1u << j) * amp;
    }
    for (int i = 0; i < (1 << r); i++) {
        uint32_t t = 0, q = 0;
        for (int m = 0; m < r; m++)
            if (i >> m & 1) {
                t |= p.reg_tmask[m];
                q |= p.reg_qmask[m];
            }
        p.reg_slot[i] = lds_slot(t) * amp;
        p.reg_qoff[i] = q;
    }
    return p;
}

// Schedule the gates of one pass onto register phases.
// Whether op h (a gate op within one layout) commutes with Z on each register
// bit of `bits`: diagonal ops do, CNOTs whose target is not in `bits` do (a Z
// on the control commutes), other one-qubit ops do unless they act on a bit
// of `bits`.
bool commutes_with_z(uint32_t h, uint32_t bits) {
    auto off = [&](uint32_t j) { return !(bits >> j & 1u); };
    if (h < H_G1 + 20) return (h - H_G1) / 5 == 3 || off((h - H_G1) % 5);
    if (h == H_RZU || (h >= H_CZ_RR && h <= H_CZ_XX) || h == H_CZG) return true;
    if (h >= H_CNOT_RR && h < H_CNOT_T) return off((h - H_CNOT_RR) / 5);
    if (h >= H_CNOT_T && h < H_CZ_RR) return off((h - H_CNOT_T) % 5);
    if (h >= H_PX && h < H_PX + 15) return (h - H_PX) / 5 == 2 || off((h - H_PX) % 5);
    return false;
}

// Register bits that op h (a gate op within one layout) changes other than
// by a diagonal factor: a CZ moves past op h when h changes none of the CZ's
// register bits (diagonal ops commute with it, and an op on other bits acts on
// other factors of the state).
uint32_t moved_bits(uint32_t h) {
    if (h < H_G1 + 20) return (h - H_G1) / 5 == 3 ? 0u : 1u << ((h - H_G1) % 5);
    if (h == H_RZU || (h >= H_CZ_RR && h <= H_CZ_XX) || h == H_DZ || h == H_CZG || (h >= H_RZN && h < H_RZN + 5))
        return 0u;
    if (h >= H_CNOT_RR && h < H_CNOT_T) return 1u << ((h - H_CNOT_RR) / 5);
    if (h >= H_CNOT_T && h < H_CZ_RR) return 1u << ((h - H_CNOT_T) % 5);
    if (h >= H_PX && h < H_PX + 15) return (h - H_PX) / 5 == 2 ? 0u : 1u << ((h - H_PX) % 5);
    if (h >= H_RYZ && h < H_RYZN + 5) return 1u << ((h - H_RYZ) % 5);
    return ~0u;
}

void schedule_pass(const std::vector<Gate>& gates, PassPlan& pp, int k, int log_r, int low,
                   uint32_t amp, std::vector<DevPhase>& phases, std::vector<DevDiag>* diags,
                   std::vector<DevFuse>* fuses, std::vector<DevCzg>* czgs) {
    const int r = log_r;
    std::vector<int> bit_of(64, -1);  // qubit -> tile bit
    for (int j = 0; j < k; j++) bit_of[pp.qubits[j]] = j;

    std::vector<int> pending = pp.gates;
    auto need_bit = [&](const Gate& g) -> int {
        int q = needed_tile_qubit(g);
        return q < 0 ? -1 : bit_of[q];
    };
    const uint32_t low_bits = (low >= 32) ? 0xffffffffu : ((1u << low) - 1);
    // gates of `pending` that one phase with register bits `regmask` runs (the
    // same ordered scan the phase itself makes)
    auto phase_gates = [&](uint32_t regmask) {
        uint64_t blocked = 0;
        int cnt = 0;
        for (int gi : pending) {
            const Gate& g = gates[gi];
            uint64_t qs = (1ull << g.q0) | (n_qubits_of(g) == 2 ? (1ull << g.q1) : 0);
            int b = need_bit(g);
            if (!(qs & blocked) && (b < 0 || (regmask >> b & 1))) cnt++;
            else blocked |= qs;
        }
        return cnt;
    };
    // Register bits of the next phase: the r allowed tile bits that let the
    // most pending gates run in that phase (all r-subsets are tried); ties
    // prefer sets without the low (coalesced) bits, so a pass more often ends
    // in a layout it can store, then the ordered-scan choice below. `forbid`
    // masks tile bits that may not be chosen.
    auto choose_scan = [&](uint32_t forbid, const std::vector<int>& keep) {
        std::vector<int> chosen;
        uint64_t blocked = 0;
        for (int gi : pending) {
            const Gate& g = gates[gi];
            uint64_t qs = (1ull << g.q0) | (n_qubits_of(g) == 2 ? (1ull << g.q1) : 0);
            if (qs & blocked) { blocked |= qs; continue; }
            int b = need_bit(g);
            if (b < 0 || std::find(chosen.begin(), chosen.end(), b) != chosen.end()) continue;
            if ((int)chosen.size() < r && !(forbid >> b & 1)) chosen.push_back(b);
            else blocked |= qs;
        }
        // fill: previous register bits first, then the lowest allowed bits
        for (int b : keep)
            if ((int)chosen.size() < r && !(forbid >> b & 1) &&
                std::find(chosen.begin(), chosen.end(), b) == chosen.end())
                chosen.push_back(b);
        for (int b = k - 1; b >= 0 && (int)chosen.size() < r; b--)
            if (!(forbid >> b & 1) && std::find(chosen.begin(), chosen.end(), b) == chosen.end())
                chosen.push_back(b);
        for (int b = k - 1; b >= 0 && (int)chosen.size() < r; b--)
            if (std::find(chosen.begin(), chosen.end(), b) == chosen.end()) chosen.push_back(b);
        std::sort(chosen.begin(), chosen.end());
        return chosen;
    };
    auto choose = [&](uint32_t forbid, const std::vector<int>& keep) {
        std::vector<int> chosen = choose_scan(forbid, keep);
        uint32_t best = 0;
        for (int b : chosen) best |= 1u << b;
        int best_n = phase_gates(best);
        bool best_low = (best & low_bits) != 0;
        for (uint32_t m = 0; m < (1u << k); m++) {
            if (__builtin_popcount(m) != r || (m & forbid)) continue;
            const int c = phase_gates(m);
            const bool lw = (m & low_bits) != 0;
            if (c > best_n || (c == best_n && best_low && !lw)) {
                best = m;
                best_n = c;
                best_low = lw;
            }
        }
        chosen.clear();
        for (int b = 0; b < k; b++)
            if (best >> b & 1) chosen.push_back(b);
        return chosen;
    };
    const uint32_t low_mask = low_bits;

    // ---- layouts. A layout is the tile bit of every register bit (`regs`,
    // by register bit) and of every thread-index bit (`thr`; bits 0-5 are lane
    // bits, the rest wavefront bits). A layout change that brings only
    // tile bits from lane bits 4 and 5 into the registers is a sequence of
    // lane swaps done in the registers (H_LSWAP, one permlane swap per
    // register pair); any other change goes through LDS (H_TRANSPOSE). Loads
    // and stores need the low tile bits on their own thread bits (thr[j] = j
    // for j < low), so lanes cover contiguous memory.
    const int log_t = k - r;
    const int home = std::min(low, log_t);
    auto swap_lane = [&](int slot) { return (slot == 4 || slot == 5) && slot < log_t; };
    auto next_use = [&](int bit) {
        int pos = 0;
        for (int gi : pending) {
            if (need_bit(gates[gi]) == bit) return pos;
            pos++;
        }
        return 1 << 30;
    };
    // thread bits for register set R after an LDS exchange: the low tile bits
    // on their own thread bits; lanes 0-3 free of them take bits of distinct
    // classes j mod 4 (the LDS slot map folds tile bit j onto slot bit j mod
    // 4, so 16 consecutive lanes then hit 16 distinct bank pairs), taken from
    // the bits needed last; the bits needed soonest on the swap lanes (4, 5);
    // the rest in order of use
    auto fresh_thr = [&](const std::vector<int>& R) {
        std::vector<int> thr(log_t, -1), rest;
        unsigned used = 0;  // classes j mod 4 on lanes 0-3
        for (int j = 0; j < k; j++) {
            if (std::find(R.begin(), R.end(), j) != R.end()) continue;
            if (j < home) {
                thr[j] = j;
                if (j < 4) used |= 1u << (j & 3);
            } else {
                rest.push_back(j);
            }
        }
        std::stable_sort(rest.begin(), rest.end(), [&](int x, int y) { return next_use(x) < next_use(y); });
        for (int sl = 0; sl < std::min(4, log_t); sl++) {
            if (thr[sl] >= 0) continue;
            for (int i = (int)rest.size() - 1; i >= 0; i--)
                if (!(used >> (rest[i] & 3) & 1)) {
                    thr[sl] = rest[i];
                    used |= 1u << (rest[i] & 3);
                    rest.erase(rest.begin() + i);
                    break;
                }
        }
        size_t ri = 0;
        for (int sl : {4, 5})
            if (swap_lane(sl) && thr[sl] < 0 && ri < rest.size()) thr[sl] = rest[ri++];
        for (int sl = 0; sl < log_t; sl++)
            if (thr[sl] < 0 && ri < rest.size()) thr[sl] = rest[ri++];
        return thr;
    };
    auto slot_of = [](const std::vector<int>& v, int bit) {
        return (int)(std::find(v.begin(), v.end(), bit) - v.begin());
    };

    std::vector<int> regs = choose(low_mask, {});
    std::vector<int> thr = fresh_thr(regs);
    // register sets reachable by lane swaps only: every incoming bit on a
    // swap lane
    auto reachable = [&](uint32_t m) {
        for (int j = 0; j < k; j++)
            if ((m >> j & 1) && std::find(regs.begin(), regs.end(), j) == regs.end() &&
                !swap_lane(slot_of(thr, j)))
                return false;
        return true;
    };
    // next register set: the best set the lane swaps reach, if it runs any
    // gate (a lane swap costs a few VALU operations per register pair, an LDS
    // exchange the whole tile's LDS traffic and two barriers); else the best
    // set overall
    auto choose_next = [&]() {
        std::vector<int> best = choose(0, regs);
        uint32_t bm = 0;
        for (int x : best) bm |= 1u << x;
        if (reachable(bm)) return best;
        int rn = 0;
        uint32_t rm = 0;
        for (uint32_t m = 0; m < (1u << k); m++) {
            if (__builtin_popcount(m) != r || !reachable(m)) continue;
            const int c = phase_gates(m);
            if (c > rn) {
                rn = c;
                rm = m;
            }
        }
        if (rn == 0) return best;
        std::vector<int> out;
        for (int j = 0; j < k; j++)
            if (rm >> j & 1) out.push_back(j);
        return out;
    };

    int cur_phase = (int)phases.size();
    phases.push_back(make_phase(pp.qubits, regs, thr, amp));
    pp.first_phase = cur_phase;

    // gradient accumulators: one per rotation in this pass
    int n_gs = 0;

    // location of qubit q in the current layout
    auto loc = [&](int q, uint32_t& type, uint32_t& pos) {
        int j = bit_of[q];
        if (j < 0) { type = LOC_FIX; pos = (uint32_t)q; return; }
        auto it = std::find(regs.begin(), regs.end(), j);
        if (it != regs.end()) { type = LOC_REG; pos = (uint32_t)(it - regs.begin()); }
        else { type = LOC_THR; pos = (uint32_t)j; }
    };
    auto make_op = [&](uint32_t h, uint32_t arg, int slot, int kind) {
        DevOp op{};
        op.h = h;
        op.arg = arg;
        op.slot = slot;
        op.kind = (uint32_t)kind;
        return op;
    };
    // bwd_arg: the argument of the op's backward form (a layout change takes
    // the backward sweep back to the previous layout)
    struct Rec { DevOp op; uint32_t bwd_arg; };
    std::vector<Rec> recs;

    // layout changes; the backward op list takes each one back to the previous layout
    auto new_phase = [&]() {
        phases.push_back(make_phase(pp.qubits, regs, thr, amp));
        return (int)phases.size() - 1;
    };
    // lane swap of register bit m and lane bit b; the argument carries the new
    // phase and the tile bits lane bit b leaves (x) and takes (y)
    auto lane_swap = [&](int m, int b) {
        const uint32_t x = (uint32_t)thr[b], y = (uint32_t)regs[m];
        std::swap(regs[m], thr[b]);
        const int np = new_phase();
        recs.push_back({make_op(H_LSWAP + (uint32_t)(m * 6 + b), lswap_arg((uint32_t)np, x, y), -1, K_H),
                        lswap_arg((uint32_t)cur_phase, y, x)});
        cur_phase = np;
        pp.n_lane_swaps++;
    };
    auto lds_exchange_to = [&](const std::vector<int>& R, const std::vector<int>& T) {
        regs = R;
        thr = T;
        const int np = new_phase();
        recs.push_back({make_op(H_TRANSPOSE, (uint32_t)np, -1, K_H), (uint32_t)cur_phase});
        cur_phase = np;
        pp.n_transposes++;
    };
    // move to register set R2: lane swaps when every incoming bit is on a
    // swap lane, else one LDS exchange
    auto change_to = [&](const std::vector<int>& R2) {
        std::vector<int> in, out;
        for (int x : R2)
            if (std::find(regs.begin(), regs.end(), x) == regs.end()) in.push_back(x);
        for (int x : regs)
            if (std::find(R2.begin(), R2.end(), x) == R2.end()) out.push_back(x);
        bool lanes = true;
        for (int x : in) lanes &= swap_lane(slot_of(thr, x));
        if (!lanes) {
            std::vector<int> R = regs;  // kept bits stay on their register bits
            for (size_t i = 0; i < out.size(); i++) R[slot_of(R, out[i])] = in[i];
            lds_exchange_to(R, fresh_thr(R));
            return;
        }
        for (size_t i = 0; i < in.size(); i++) lane_swap(slot_of(regs, out[i]), slot_of(thr, in[i]));
    };

    // RZ groups: within the ops of one layout, each RZ on a register bit is
    // moved later, past ops that commute with it (an RZ and its gradient term
    // are unchanged by that), and collected. An op that does not commute with
    // a collected RZ, or a second RZ on its bit, ends the collection there:
    // as one H_DZ op if MIN_DZ_SIZE or more RZs are collected, else by putting
    // out only the RZs in the way, on their own (the others move on).
    auto group_rz = [&](size_t seg0) {
        if (!diags || r > MAX_DZ_BITS) return;
        std::vector<Rec> out(recs.begin(), recs.begin() + (long)seg0);
        Rec grp[MAX_DZ_BITS];
        uint32_t bits = 0;
        auto put_out = [&](uint32_t which) {
            if (__builtin_popcount(bits) >= MIN_DZ_SIZE) {
                DevDiag d;
                for (int j = 0; j < MAX_DZ_BITS; j++) {
                    d.slot[j] = (bits >> j & 1u) ? grp[j].op.slot : -1;
                    d.gslot[j] = (bits >> j & 1u) ? grp[j].op.arg : NO_GSLOT;
                }
                const uint32_t idx = (uint32_t)diags->size();
                diags->push_back(d);
                out.push_back({make_op(H_DZ, idx, -1, K_RZ), idx});
                bits = 0;
                return;
            }
            for (int j = 0; j < MAX_DZ_BITS; j++)
                if ((which & bits) >> j & 1u) out.push_back(grp[j]);
            bits &= ~which;
        };
        for (size_t i = seg0; i < recs.size(); i++) {
            const uint32_t h = recs[i].op.h;
            if (h >= H_G1 + 15 && h < H_G1 + 15 + (uint32_t)r) {
                const uint32_t j = h - (H_G1 + 15);
                if (bits >> j & 1u) put_out(1u << j);
                grp[j] = recs[i];
                bits |= 1u << j;
                continue;
            }
            uint32_t clash = 0;
            for (int j = 0; j < MAX_DZ_BITS; j++)
                if ((bits >> j & 1u) && !commutes_with_z(h, 1u << j)) clash |= 1u << j;
            if (clash) put_out(clash);
            out.push_back(recs[i]);
        }
        put_out(bits);
        recs.swap(out);
    };
    // RY-RZ pairs: an RZ left on its own after grouping joins the nearest
    // earlier RY on its register bit in the same layout when every op between
    // them commutes with Z on that bit (the RZ moves back to the RY); the pair
    // runs as one H_RYZ op.
    auto pair_ryz = [&](size_t seg0) {
        if (!fuses) return;
        std::vector<bool> gone(recs.size(), false);
        for (size_t i = seg0; i < recs.size(); i++) {
            const uint32_t h = recs[i].op.h;
            if (!(h >= H_G1 + 15 && h < H_G1 + 15 + (uint32_t)r)) continue;
            const uint32_t j = h - (H_G1 + 15);
            for (size_t k = i; k-- > seg0;) {
                if (gone[k]) continue;
                const uint32_t hk = recs[k].op.h;
                if (hk == H_G1 + 10 + j) {
                    if (fuses->size() >= 65536) break;
                    const uint32_t idx = (uint32_t)fuses->size();
                    fuses->push_back({recs[i].op.slot, recs[i].op.arg});
                    const uint32_t arg = recs[k].op.arg | recs[i].op.arg << 8 | idx << 16;
                    recs[k].op.h = H_RYZ + j;
                    recs[k].op.arg = arg;
                    recs[k].bwd_arg = arg;
                    gone[i] = true;
                    break;
                }
                if (!commutes_with_z(hk, 1u << j)) break;
            }
        }
        std::vector<Rec> out;
        for (size_t i = 0; i < recs.size(); i++)
            if (!gone[i]) out.push_back(recs[i]);
        recs.swap(out);
    };

    // CZ groups: within the ops of one layout, each CZ moves later, past ops
    // that change none of its register bits (see moved_bits), and is
    // collected. An op that changes a register bit of a collected CZ puts out
    // every collected CZ before it (each has moved only past ops it commutes
    // with), two or more as one H_CZG op; so does the end of the layout. A
    // ring of CZs between two rotation layers becomes one op.
    auto cz_reg_bits = [](uint32_t h) -> uint32_t {
        if (h >= H_CZ_RR && h < H_CZ_RX) return (1u << ((h - H_CZ_RR) / 5)) | (1u << ((h - H_CZ_RR) % 5));
        if (h >= H_CZ_RX && h < H_CZ_XX) return 1u << (h - H_CZ_RX);
        return 0u;
    };
    auto group_cz = [&](size_t seg0) {
        if (!czgs || r > CZG_REG_BITS) return;
        std::vector<Rec> out(recs.begin(), recs.begin() + (long)seg0);
        std::vector<Rec> grp;
        auto emit = [&](const std::vector<Rec>& g) {
            if (g.size() == 1) out.push_back(g[0]);
            if (g.size() < 2) return;
            DevCzg d{};
            uint32_t tt[MAX_CZG_PAIRS], other[MAX_CZG_PAIRS], n_tt = 0, n_other = 0;
            auto flush = [&]() {
                for (uint32_t i = 0; i < n_tt; i++) d.pair[i] = tt[i];
                for (uint32_t i = 0; i < n_other; i++) d.pair[n_tt + i] = other[i];
                d.n_tt = n_tt;
                d.n_pairs = n_tt + n_other;
                const uint32_t idx = (uint32_t)czgs->size();
                czgs->push_back(d);
                out.push_back({make_op(H_CZG, idx, -1, K_CZ), idx});
                d = DevCzg{};
                n_tt = n_other = 0;
            };
            for (const Rec& rc : g) {
                const uint32_t h = rc.op.h, w = rc.op.arg;
                if (h >= H_CZ_RR && h < H_CZ_RX) {
                    const uint32_t a = (h - H_CZ_RR) / 5, b = (h - H_CZ_RR) % 5;
                    for (uint32_t i = 0; i < (1u << r); i++)
                        if ((i >> a & 1u) && (i >> b & 1u)) d.reg_mask ^= 1u << i;
                } else if (h >= H_CZ_RX && h < H_CZ_XX) {
                    const uint32_t a = h - H_CZ_RX, pos = w & 0xff;
                    if (((w >> 8) & 3) == LOC_THR) d.thr[a] ^= 1u << pos;
                    else d.fix[a] ^= 1u << pos;
                } else {
                    if (n_tt + n_other == MAX_CZG_PAIRS) flush();
                    uint32_t wa = w & 0xffff, wb = w >> 16;
                    if (((wa >> 8) & 3) != LOC_THR) std::swap(wa, wb);  // a thread operand first
                    if (((wb >> 8) & 3) == LOC_THR) tt[n_tt++] = (wa & 0xff) | (wb & 0xff) << 8;
                    else other[n_other++] = wa | wb << 16;
                }
            }
            flush();
        };
        for (size_t i = seg0; i < recs.size(); i++) {
            const uint32_t h = recs[i].op.h;
            if (h >= H_CZ_RR && h <= H_CZ_XX) {
                grp.push_back(recs[i]);
                continue;
            }
            const uint32_t mv = moved_bits(h);
            uint32_t clash = 0;
            for (const Rec& rc : grp) clash |= cz_reg_bits(rc.op.h) & mv;
            if (clash || mv == ~0u) {
                emit(grp);
                grp.clear();
            }
            out.push_back(recs[i]);
        }
        emit(grp);
        recs.swap(out);
    };

    while (!pending.empty()) {
        uint64_t blocked = 0;
        std::vector<int> rest;
        const size_t seg0 = recs.size();
        for (int gi : pending) {
            const Gate& g = gates[gi];
            uint64_t qs = (1ull << g.q0) | (n_qubits_of(g) == 2 ? (1ull << g.q1) : 0);
            int b = need_bit(g);
            bool ok = !(qs & blocked) &&
                      (b < 0 || std::find(regs.begin(), regs.end(), b) != regs.end());
            if (!ok) { blocked |= qs; rest.push_back(gi); continue; }
            uint32_t gs = NO_GSLOT;
            if (is_rotation(g.kind)) {
                gs = (uint32_t)n_gs++;
                pp.gslots.push_back(g.slot);
            }
            uint32_t ta, pa, tb, pb;
            DevOp op{};
            switch (g.kind) {
                case K_PAULI:  // planned on a register bit, like RX
                    loc(g.q0, ta, pa);
                    op = make_op(H_PX + pa, 0, g.slot, K_PAULI);
                    break;
                case K_H: case K_RX: case K_RY: case K_RZ:
                    loc(g.q0, ta, pa);
                    if (ta == LOC_REG)
                        op = make_op(H_G1 + (uint32_t)(g.kind * 5 + (int)pa), gs, g.slot, g.kind);
                    else  // only RZ reaches here: diagonal, no register bit needed
                        op = make_op(H_RZU, loc_word(ta, pa) | (gs << 16), g.slot, g.kind);
                    break;
                case K_CNOT:
                    loc(g.q1, ta, pa);  // target: always a register bit here
                    loc(g.q0, tb, pb);
                    if (tb == LOC_REG) op = make_op(H_CNOT_RR + pa * 5 + pb, 0, -1, K_CNOT);
                    else if (tb == LOC_THR) op = make_op(H_CNOT_T + pa, pb, -1, K_CNOT);
                    else op = make_op(H_CNOT_F + pa, pb, -1, K_CNOT);
                    break;
                case K_CZ:
                    loc(g.q0, ta, pa);
                    loc(g.q1, tb, pb);
                    if (ta != LOC_REG && tb == LOC_REG) {
                        std::swap(ta, tb);
                        std::swap(pa, pb);
                    }
                    if (ta == LOC_REG && tb == LOC_REG) op = make_op(H_CZ_RR + pa * 5 + pb, 0, -1, K_CZ);
                    else if (ta == LOC_REG) op = make_op(H_CZ_RX + pa, loc_word(tb, pb), -1, K_CZ);
                    else op = make_op(H_CZ_XX, loc_word(ta, pa) | (loc_word(tb, pb) << 16), -1, K_CZ);
                    break;
            }
            recs.push_back({op, op.arg});
        }
        group_rz(seg0);
        pair_ryz(seg0);
        group_cz(seg0);
        pending.swap(rest);
        if (pending.empty()) break;
        change_to(choose_next());
    }
    // end in a store layout: the low tile bits back on their own thread bits
    // (through LDS if any has left them)
    bool fits = true;
    for (int j = 0; j < home; j++) fits &= thr[j] == j;
    if (!fits) {
        std::vector<int> keep;
        for (int x : regs)
            if (x >= home) keep.push_back(x);
        pending.clear();
        std::vector<int> R = choose_scan(low_mask, keep);
        lds_exchange_to(R, fresh_thr(R));
    }
    pp.last_phase = cur_phase;
    for (auto& rc : recs) pp.fwd_ops.push_back(rc.op);
    for (int i = (int)recs.size() - 1; i >= 0; i--) {
        DevOp op = recs[i].op;
        op.arg = recs[i].bwd_arg;
        pp.bwd_ops.push_back(op);
    }
    // A backward layout change refreshes the thread's Im<lambda|psi> sum only
    // when an RZ-type gradient term (RZ on a register, thread or fixed bit,
    // an RZ group, an RY-RZ pair) reads it before the next layout change.
    auto layout_change = [](uint32_t h) { return h == H_TRANSPOSE || (h >= H_LSWAP && h < H_PX); };
    auto reads_ival = [](uint32_t h) {
        return (h >= H_G1 + 15 && h < H_G1 + 20) || h == H_RZU || (h >= H_RZN && h < H_RZN + 5) || h == H_DZ ||
               (h >= H_RYZ && h < H_RYZN + 5);
    };
    for (size_t i = 0; i < pp.bwd_ops.size(); i++) {
        if (!layout_change(pp.bwd_ops[i].h)) continue;
        for (size_t j = i + 1; j < pp.bwd_ops.size() && !layout_change(pp.bwd_ops[j].h); j++)
            if (reads_ival(pp.bwd_ops[j].h)) {
                pp.bwd_ops[i].arg |= ARG_IVAL;
                break;
            }
    }
}

}  // namespace

int whole_state_max_qubits(int dtype) { return dtype == 0 ? 12 : 11; }

std::string build_circuit(int n, const int32_t* g5, int n_gates, int n_inputs, int n_weights,
                          const Extras& ext, const Options& opts, Circuit& out) {
    if (n < 1 || n > 32) return fmt("n_qubits=%ld out of range [1, 32]", n);
    if (n_gates < 0) return "n_gates < 0";
    if (n_gates > 0 && !g5) return "gates is NULL";
    if (n_inputs < 0 || n_weights < 0) return "negative n_inputs or n_weights";
    if (n_gates > (1 << 22)) return "too many gates";
    out = Circuit{};
    out.n = n;
    out.n_inputs = n_inputs;
    out.n_weights = n_weights;
    out.n_user_gates = n_gates;
    out.opts = opts;
    out.embed = ext.embed;
    out.embed_first = ext.embed_first;
    if (ext.embed == E_BASIS) {
        if (ext.embed_first < 0 || (int64_t)ext.embed_first + n > n_inputs)
            return fmt("basis embedding needs features [%ld, %ld + n) within n_inputs = %ld", ext.embed_first,
                       ext.embed_first, n_inputs);
    } else if (ext.embed == E_AMPLITUDE) {
        if (n > AMPLITUDE_MAX_QUBITS) return fmt("amplitude embedding supports at most %ld qubits", AMPLITUDE_MAX_QUBITS);
        if (ext.embed_first < 0 || (int64_t)ext.embed_first + ((int64_t)1 << n) > n_inputs)
            return fmt("amplitude embedding needs features [%ld, %ld + 2^n) within n_inputs = %ld",
                       ext.embed_first, ext.embed_first, n_inputs);
    } else if (ext.embed != E_NONE) {
        return fmt("unknown embedding %ld", ext.embed);
    }
    // rotation occurrences in gate order; numbered below (trainable first)
    std::vector<Slot> pending_slots;
    std::vector<int> slot_of_gate;  // per internal gate: pending slot or -1
    int user = 0;                   // gate as given being rewritten
    auto emit = [&](int kind, int q0, int q1, const Slot* sl) {
        out.gates.push_back(Gate{kind, q0, q1, sl ? sl->src : (int)S_NONE, sl ? sl->index : 0, -1, user});
        slot_of_gate.push_back(sl ? (int)pending_slots.size() : -1);
        if (sl) pending_slots.push_back(*sl);
    };
    int n_channels = 0;
    for (int i = 0; i < n_gates; i++) {
        user = i;
        const int kind = g5[5 * i], q0 = g5[5 * i + 1], q1 = g5[5 * i + 2], src = g5[5 * i + 3],
                  index = g5[5 * i + 4];
        if (kind < K_H || kind > P_PAULI) return fmt("gate %ld: unknown kind %ld", i, kind);
        if (q0 < 0 || q0 >= n) return fmt("gate %ld: qubit %ld out of range", i, q0);
        const bool two = kind == K_CNOT || kind == K_CZ || kind == P_CRX || kind == P_CRY || kind == P_CRZ;
        if (two) {
            if (q1 < 0 || q1 >= n) return fmt("gate %ld: qubit %ld out of range", i, q1);
            if (q1 == q0) return fmt("gate %ld: q0 == q1 == %ld", i, q0);
        } else if (q1 != -1) {
            return fmt("gate %ld: one-qubit gate needs q1 = -1 (got %ld)", i, q1);
        }
        const bool angled = is_rotation(kind) || kind == P_CRX || kind == P_CRY || kind == P_CRZ;
        if (angled) {
            if (src == S_INPUT) {
                if (index < 0 || index >= n_inputs)
                    return fmt("gate %ld: input index %ld out of range [0, %ld)", i, index, n_inputs);
            } else if (src == S_WEIGHT) {
                if (index < 0 || index >= n_weights)
                    return fmt("gate %ld: weight index %ld out of range [0, %ld)", i, index, n_weights);
            } else {
                return fmt("gate %ld: rotation needs src INPUT or WEIGHT (got %ld)", i, src);
            }
        } else if (kind == P_PAULI) {
            if (src != S_INPUT || index < 0 || index >= n_inputs)
                return fmt("gate %ld: Pauli channel needs src INPUT and an input index in [0, %ld)", i, n_inputs);
        } else if (src != S_NONE) {
            return fmt("gate %ld: H/CNOT/CZ take no angle source (got %ld)", i, src);
        }
        if (kind <= K_CZ) {
            Slot sl{src, index, 1.0, 0, 0, 0};
            emit(kind, q0, q1, is_rotation(kind) ? &sl : nullptr);
        } else if (kind == P_PAULI) {
            if (!ext.pauli_p) return fmt("gate %ld: Pauli channel without probabilities", i);
            const double* p = ext.pauli_p + 3 * n_channels++;
            if (!(p[0] >= 0 && p[1] >= 0 && p[2] >= 0 && p[0] + p[1] + p[2] <= 1.0))
                return fmt("gate %ld: Pauli probabilities must be >= 0 with sum <= 1", i);
            const Slot sl{S_PAULI, index, 1.0, p[0], p[0] + p[1], p[0] + p[1] + p[2]};
            if (p[0] > 0 || p[1] > 0 || p[2] > 0) emit(K_PAULI, q0, -1, &sl);
        } else {
            // controlled rotation CR(t) on (control q0, target q1) as
            // R(t/2) E R(-t/2) E with E = CNOT(q0, q1) for RY and RZ (X R(a) X =
            // R(-a)) and E = CZ(q0, q1) for RX (Z RX(a) Z = RX(-a))
            const int rot = kind == P_CRX ? K_RX : kind == P_CRY ? K_RY : K_RZ;
            const int ent = kind == P_CRX ? K_CZ : K_CNOT;
            Slot hp{src, index, 0.5, 0, 0, 0}, hm{src, index, -0.5, 0, 0, 0};
            emit(rot, q1, -1, &hp);
            emit(ent, q0, q1, nullptr);
            emit(rot, q1, -1, &hm);
            emit(ent, q0, q1, nullptr);
        }
    }
    // slot numbers: input/weight slots in gate order, then Pauli slots
    std::vector<int> num(pending_slots.size(), -1);
    for (int pass = 0; pass < 2; pass++)
        for (size_t s = 0; s < pending_slots.size(); s++)
            if ((pending_slots[s].src == S_PAULI) == (pass == 1)) {
                num[s] = (int)out.slots.size();
                out.slots.push_back(pending_slots[s]);
                if (pass == 0) out.n_param_slots++;
            }
    for (size_t i = 0; i < out.gates.size(); i++)
        if (slot_of_gate[i] >= 0) out.gates[i].slot = num[slot_of_gate[i]];
    const Options& o = opts;
    if (o.log_regs && (o.log_regs < 2 || o.log_regs > MAX_LOG_R)) return "option: log_regs out of range [2, 5]";
    if (o.log_threads && (o.log_threads < 6 || o.log_threads > 9)) return "option: log_threads out of range [6, 9]";
    if (o.low_qubits && (o.low_qubits < 1 || o.low_qubits > 8)) return "option: low_qubits out of range [1, 8]";
    if (o.max_gates_per_pass < 0) return "option: max_gates_per_pass < 0";
    if (o.wg_per_sample < 0) return "option: wg_per_sample < 0";
    if (o.rz_groups != 0 && o.rz_groups != -1) return "option: rz_groups must be 0 or -1";
    if (o.cz_groups != 0 && o.cz_groups != -1) return "option: cz_groups must be 0 or -1";
    if (o.product_prefix < -1 || o.product_prefix > 1) return "option: product_prefix must be -1, 0 or 1";
    if (o.pass_search < -1 || o.pass_search > 1) return "option: pass_search must be -1, 0 or 1";
    for (int dt = 0; dt < 2; dt++) {
        std::string e = build_plan(out, dt, out.plan[dt]);
        if (!e.empty()) return e;
    }
    return "";
}

std::string build_plan(const Circuit& c, int dtype, Plan& pl) {
    pl = Plan{};
    pl.n = c.n;
    pl.n_slots = (int)c.slots.size();
    const Options& o = c.opts;
    // The register-tile kernel needs at least 2^8 amplitudes per tile; below
    // that, or when asked (force_tiled < 0) and the state fits in LDS, the
    // whole state of a sample lives in one workgroup's LDS.
    if (c.n < 8 || (o.force_tiled < 0 && c.n <= whole_state_max_qubits(dtype))) {
        pl.whole_state = true;
        PassPlan pp;
        for (int i = 0; i < (int)c.gates.size(); i++) pp.gates.push_back(i);
        for (int q = 0; q < c.n; q++) pp.qubits.push_back(q);
        pl.passes.push_back(pp);
        pl.k = c.n;
        return "";
    }
    // complex64: 16 amplitudes per thread and 512 threads (a 2^13-amplitude
    // tile, four wavefronts per SIMD); complex128: 16 per thread, 256 threads
    int log_r = o.log_regs ? o.log_regs : 4;
    int log_t = o.log_threads ? o.log_threads : (dtype == 0 ? 9 : 8);
    // A circuit smaller than the default tile runs one tile per sample; such
    // passes are latency-bound, so unless asked otherwise the tile keeps its
    // threads (more wavefronts per sample) and gives up registers first.
    if (!o.log_regs)
        while (log_r + log_t > c.n && log_r > 2) log_r--;
    while (log_r + log_t > c.n && log_t > 6) log_t--;
    while (log_r + log_t > c.n && log_r > 2) log_r--;
    if (log_r + log_t > c.n) return "circuit too small for the tile kernel";
    const int k = log_r + log_t;
    int low = o.low_qubits ? o.low_qubits : (dtype == 0 ? 4 : 3);
    if (low > k - 1) low = k - 1;
    if (c.n == k) low = k;
    pl.k = k;
    pl.log_r = log_r;
    pl.log_t = log_t;
    pl.low = low;

    const int G = (int)c.gates.size();
    std::vector<char> done(G, 0);
    int remaining = G;
    // Product prefix: a one-qubit gate on a qubit that no two-qubit gate or
    // Pauli channel has touched yet commutes with every earlier gate on other
    // qubits, so all such gates can run first, on |0...0>, where they make a
    // product state. They leave the passes (marked done for the planner).
    std::vector<int> pre_gates;
    std::vector<std::vector<DevPrefix>> per(c.n);
    if (c.embed == E_NONE && o.product_prefix >= 0) {
        uint64_t touched = 0;
        for (int i = 0; i < G; i++) {
            const Gate& g = c.gates[i];
            if (n_qubits_of(g) == 2) {
                touched |= (1ull << g.q0) | (1ull << g.q1);
            } else if (g.kind == K_PAULI) {
                touched |= 1ull << g.q0;
            } else if (!(touched >> g.q0 & 1)) {
                per[g.q0].push_back({g.kind, g.slot});
                pre_gates.push_back(i);
            }
        }
    }
    const uint64_t low_tile = (low >= 64) ? ~0ull : ((1ull << low) - 1);
    // Candidate tiles of the next pass: first-need greedy growth, and
    // contiguous windows of the high qubits.
    struct Cand {
        std::vector<int> gates;
        uint64_t tile;
    };
    auto candidates = [&](const std::vector<char>& dn) {
        std::vector<Cand> out;
        uint64_t t = low_tile;
        std::vector<int> e = scan(c.gates, dn, t, k, true, o.max_gates_per_pass);
        out.push_back({std::move(e), t});
        const int h = k - low;
        for (int s = low; s + h <= c.n; s++) {
            uint64_t w = low_tile | (((1ull << h) - 1) << s);
            std::vector<int> ew = scan(c.gates, dn, w, k, false, o.max_gates_per_pass);
            out.push_back({std::move(ew), w});
        }
        return out;
    };
    // the candidate that executes the most gates (the first of equals)
    auto widest = [](const std::vector<Cand>& cs) {
        size_t b = 0;
        for (size_t i = 1; i < cs.size(); i++)
            if (cs[i].gates.size() > cs[b].gates.size()) b = i;
        return b;
    };
    // Cost model of the look-ahead, in FMAs per amplitude. A pass is bound by
    // its memory traffic or by its arithmetic, whichever takes longer: a
    // forward pass moves 2 amplitudes (16 B in complex64) per amplitude and
    // does 3 FMAs per rotation (RX, RY); a backward pass moves 3 (psi and
    // lambda in, lambda out) and does 8 per rotation (psi and lambda
    // un-applied, the gradient term). At about 5 TB/s of streaming bandwidth
    // against about 3.8e13 fp32 FMA/s (MI355X), one byte costs as long as 7.6
    // FMAs. Other gates count by their arithmetic relative to a rotation.
    const double amp_bytes = dtype == 0 ? 8.0 : 16.0;
    const double mem_fwd = 7.6 * 2 * amp_bytes, mem_bwd = 7.6 * 3 * amp_bytes;
    auto weight = [&](const std::vector<int>& ex) {
        double w = 0;
        for (int i : ex) {
            const int kd = c.gates[i].kind;
            w += (kd == K_RX || kd == K_RY) ? 1.0 : kd == K_RZ ? 0.5 : kd == K_H ? 0.7 : 0.25;
        }
        return w;
    };
    auto pass_cost = [&](double w) { return std::max(mem_fwd, 3 * w) + std::max(mem_bwd, 8 * w); };
    // Greedy completion from `dn` for at most `horizon` passes; the gates
    // left after it are priced at their arithmetic alone.
    auto rollout = [&](std::vector<char> dn, int rem, int horizon) {
        double cost = 0;
        for (int p = 0; p < horizon && rem > 0; p++) {
            std::vector<Cand> cs = candidates(dn);
            const Cand& b = cs[widest(cs)];
            if (b.gates.empty()) return 1e300;
            for (int i : b.gates) dn[i] = 1;
            rem -= (int)b.gates.size();
            cost += pass_cost(weight(b.gates));
        }
        if (rem > 0) {
            std::vector<int> left;
            for (int i = 0; i < G; i++)
                if (!dn[i]) left.push_back(i);
            cost += 11 * weight(left);
        }
        return cost;
    };
    // The look-ahead's rollouts cost about horizon x candidates^2 x gates per
    // pass, the beam search width x candidates x gates per depth; both are
    // sized from the greedy plan's pass count so that planning stays within
    // a fraction of a second (full look-aheads and a beam of 64 for the
    // workloads' circuits, shorter and narrower ones for plans of many passes).
    int horizon = 32, width = 64;
    // Beam search over whole pass sequences: each depth extends every kept
    // partial plan by every candidate tile, keeps the `width` distinct ones
    // that leave the fewest gates (ties: least modeled cost), and stops at the
    // first depth where a plan is complete, returning up to 8 complete plans,
    // cheapest first.
    auto beam_search = [&](int width) {
        struct St {
            std::vector<char> dn;
            int rem;
            double cost;
            std::vector<Cand> seq;
        };
        std::vector<St> beam{{done, remaining, 0.0, {}}};
        for (;;) {
            std::vector<St> next;
            for (const St& s : beam)
                for (Cand& cd : candidates(s.dn)) {
                    if (cd.gates.empty()) continue;
                    St ns{s.dn, s.rem - (int)cd.gates.size(), s.cost + pass_cost(weight(cd.gates)), s.seq};
                    for (int g : cd.gates) ns.dn[g] = 1;
                    ns.seq.push_back(std::move(cd));
                    next.push_back(std::move(ns));
                }
            if (next.empty()) return std::vector<std::vector<Cand>>();
            std::stable_sort(next.begin(), next.end(), [](const St& a, const St& b) {
                return a.rem != b.rem ? a.rem < b.rem : a.cost < b.cost;
            });
            if (next[0].rem == 0) {  // the complete plans of this depth, cheapest first
                std::vector<std::vector<Cand>> done_plans;
                for (St& s : next)
                    if (s.rem == 0 && done_plans.size() < 8) done_plans.push_back(std::move(s.seq));
                return done_plans;
            }
            std::vector<St> kept;
            std::set<std::vector<char>> seen;
            for (St& s : next) {
                if ((int)kept.size() >= width) break;
                if (seen.insert(s.dn).second) kept.push_back(std::move(s));
            }
            beam = std::move(kept);
        }
    };
    // One pass at a time: the greedy choice is the candidate that executes
    // the most gates; the look-ahead prices each candidate by the cost of its
    // pass plus a greedy completion of the rest of the circuit, which avoids
    // a tail of nearly empty, memory-bound passes (such as the ends of long
    // CNOT chains).
    auto one_at_a_time = [&](bool look) {
        std::vector<Cand> seq;
        std::vector<char> dn = done;
        int rem = remaining;
        while (rem > 0) {
            std::vector<Cand> cs = candidates(dn);
            size_t pick = widest(cs);
            if (look) {
                double best_cost = 1e300;
                for (size_t i = 0; i < cs.size(); i++) {
                    if (cs[i].gates.empty()) continue;
                    std::vector<char> d2 = dn;
                    for (int g : cs[i].gates) d2[g] = 1;
                    const double cst = pass_cost(weight(cs[i].gates)) +
                                       rollout(std::move(d2), rem - (int)cs[i].gates.size(), horizon);
                    if (cst < best_cost * (1 - 1e-12) ||
                        (cst <= best_cost * (1 + 1e-12) && cs[i].gates.size() > cs[pick].gates.size())) {
                        best_cost = cst;
                        pick = i;
                    }
                }
            }
            if (cs[pick].gates.empty()) return std::vector<Cand>();
            for (int g : cs[pick].gates) dn[g] = 1;
            rem -= (int)cs[pick].gates.size();
            seq.push_back(std::move(cs[pick]));
        }
        return seq;
    };
    // Lay out a pass sequence: each pass's register phases, exchanges and ops.
    auto lay_out = [&](std::vector<Cand> seq, Plan& to) {
        for (Cand& cd : seq) {
            uint64_t tile = cd.tile;
            // fill the tile up to k qubits with the lowest unused qubits
            for (int q = 0; q < c.n && __builtin_popcountll(tile) < k; q++) tile |= 1ull << q;
            PassPlan pp;
            for (int q = 0; q < c.n; q++) if (tile >> q & 1) pp.qubits.push_back(q);
            pp.gates = std::move(cd.gates);
            schedule_pass(c.gates, pp, k, log_r, low, dtype == 0 ? 8u : 16u, to.phases,
                          o.rz_groups == 0 ? &to.diags : nullptr, o.rz_groups == 0 ? &to.fuses : nullptr,
                          o.cz_groups == 0 ? &to.czgs : nullptr);
            to.passes.push_back(std::move(pp));
        }
    };
    // By default the plans of fewest passes among the look-ahead's and the
    // beam search's complete plans are laid out, and the one with the fewest
    // layout changes is taken (an LDS exchange weighed as three lane swaps):
    // 30q: 9 passes against the look-ahead's 11, 24q: 14 against 15. Plans
    // the remaining gates (those not marked done) into `to`; returns its
    // layout score, or -1 when the planner makes no progress.
    auto choose = [&](Plan& to) -> int {
        std::vector<std::vector<Cand>> plans;
        if (remaining > 0) {
            plans.push_back(one_at_a_time(false));
            if (plans[0].empty()) return -1;
            const double nc = (double)candidates(done).size();
            const double unit = (double)plans[0].size() * nc * std::max(G, 1);
            horizon = (int)std::max(2.0, std::min(32.0, 2e8 / (unit * nc)));
            width = (int)std::max(4.0, std::min(64.0, 1e8 / unit));
            if (o.pass_search != -1) plans[0] = one_at_a_time(true);
            if (plans[0].empty()) return -1;
            if (o.pass_search == 0) {
                std::vector<std::vector<Cand>> bs = beam_search(width);
                if (!bs.empty() && bs[0].size() < plans[0].size()) plans.clear();
                for (auto& p : bs)
                    if (p.size() == (plans.empty() ? bs[0].size() : plans[0].size())) plans.push_back(std::move(p));
            }
        } else {
            plans.push_back({{{}, low_tile}});  // no gates: one empty pass
        }
        int best = -1;
        for (auto& p : plans) {
            Plan t;
            lay_out(std::move(p), t);
            int score = 0;
            for (const PassPlan& pp : t.passes) score += 3 * pp.n_transposes + pp.n_lane_swaps;
            if (best < 0 || score < best) {
                best = score;
                to.passes = std::move(t.passes);
                to.phases = std::move(t.phases);
                to.diags = std::move(t.diags);
                to.fuses = std::move(t.fuses);
                to.czgs = std::move(t.czgs);
            }
        }
        return best;
    };
    // The product prefix takes its gates out of the passes. By default it is
    // kept when the rest of the circuit then needs fewer passes, or as many
    // passes and no more layout changes (30q: 9 passes either way, 24
    // exchanges and 72 lane swaps against 26 and 76; 16q: 5 passes against
    // 6); otherwise (24q: 41 exchanges against 35) the op plan is kept and
    // only the prefix gates of its first pass form the product state.
    // product_prefix = 1 keeps the whole prefix always, -1 never.
    const int score_ops = choose(pl);
    if (score_ops < 0) return "planner made no progress";
    // take plan t with the prefix gates `absorbed` (each qubit's a leading run
    // of its prefix) as the initial product state
    auto take = [&](Plan& t, const std::vector<int>& absorbed) {
        pl.passes = std::move(t.passes);
        pl.phases = std::move(t.phases);
        pl.diags = std::move(t.diags);
        pl.fuses = std::move(t.fuses);
        pl.czgs = std::move(t.czgs);
        pl.product = true;
        pl.pre_gates = absorbed;
        std::vector<std::vector<DevPrefix>> mine(c.n);
        for (int i : absorbed) mine[c.gates[i].q0].push_back({c.gates[i].kind, c.gates[i].slot});
        pl.pre_ptr.assign(1, 0);
        pl.pre_ops.clear();
        for (int q = 0; q < c.n; q++) {
            pl.pre_ops.insert(pl.pre_ops.end(), mine[q].begin(), mine[q].end());
            pl.pre_ptr.push_back((int32_t)pl.pre_ops.size());
        }
    };
    if (!pre_gates.empty()) {
        for (int i : pre_gates) done[i] = 1;
        remaining -= (int)pre_gates.size();
        Plan t;
        const int score_pre = choose(t);
        if (score_pre >= 0 && (o.product_prefix == 1 || t.passes.size() < pl.passes.size() ||
                               (t.passes.size() == pl.passes.size() && score_pre <= score_ops))) {
            take(t, pre_gates);
        } else if (o.product_prefix == 0 && !pl.passes.empty()) {
            // Otherwise the prefix gates the first pass of the op plan runs
            // anyway (a leading run of each of its qubits' prefixes) become
            // its initial product state; the passes stay as they are.
            std::vector<char> in0(G, 0);
            for (int i : pl.passes[0].gates) in0[i] = 1;
            std::vector<char> take0(G, 0);
            std::vector<int> absorbed;
            std::vector<int> by_q(c.n, 0);
            for (int i : pre_gates) {  // gate order: per qubit, stop at the first one pass 0 lacks
                const int q = c.gates[i].q0;
                if (by_q[q] < 0) continue;
                if (in0[i]) {
                    take0[i] = 1;
                    absorbed.push_back(i);
                } else {
                    by_q[q] = -1;
                }
            }
            if (!absorbed.empty()) {
                std::vector<Cand> seq;
                for (const PassPlan& pp : pl.passes) {
                    Cand cd;
                    cd.tile = 0;
                    for (int q : pp.qubits) cd.tile |= 1ull << q;
                    for (int i : pp.gates)
                        if (!take0[i]) cd.gates.push_back(i);
                    seq.push_back(std::move(cd));
                }
                Plan t2;
                lay_out(std::move(seq), t2);
                int score = 0;
                for (const PassPlan& pp : t2.passes) score += 3 * pp.n_transposes + pp.n_lane_swaps;
                if (score <= score_ops) take(t2, absorbed);
            }
        }
    }
    if (pl.phases.size() > 65535) return "plan too large (phases)";
    return "";
}

}  // namespace qlayer
