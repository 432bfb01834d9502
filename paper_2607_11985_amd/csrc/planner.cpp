// planner.cpp -- compile phase (Algorithm 1, compile phase): validate the
// static gate list, lower it to primitives, classify every angle as parametric
// (param / input slot) or constant (cached cos/sin), and plan the register-tile
// schedules of the forward sweep and of the adjoint (reverse) sweep.
//
// Resident path (n <= 13 by default): one pass holds every qubit on chip.
// Streaming path (n >= 14): a pass holds k "local" qubits of one sample in a
// workgroup (k = 12, 13 or 14); the other ng = n - k "global" qubits are fixed
// per workgroup (its tile index).  A pass runs every gate whose qubit lines are
// ready and whose register-bit qubit is local -- gates on disjoint qubits
// commute, so a gate that must wait blocks only its own lines.  Diagonal gates
// and CNOT controls may sit on global qubits (their value is uniform over the
// tile).
//
// Host-only code: no device calls, so it can run (and be tested) without a GPU.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <map>
#include <set>

#include "vqc.h"
#include "vqc_internal.h"

static_assert(vqc::kSrcParam == VQC_SRC_PARAM && vqc::kSrcInput == VQC_SRC_INPUT &&
                  vqc::kSrcConst == VQC_SRC_CONST,
              "angle source codes of the device header and the C ABI differ");
static_assert(vqc::kLossSum == VQC_LOSS_SUM && vqc::kLossMean == VQC_LOSS_MEAN &&
                  vqc::kLossMseZ0 == VQC_LOSS_MSE_Z0 && vqc::kLossMseMeanZ == VQC_LOSS_MSE_MEANZ,
              "loss head codes of the device header and the C ABI differ");

namespace vqc {
namespace {

struct Mapping {
  int k = 0, nq = 0;
  int p2q[kMaxTileQubits];  // local physical bit -> logical qubit
  int q2p[kMaxQubits];      // logical qubit -> physical bit (>= k: global bit + k)
  bool operator==(const Mapping& o) const {
    return k == o.k && nq == o.nq && std::memcmp(p2q, o.p2q, sizeof(int) * k) == 0 &&
           std::memcmp(q2p, o.q2p, sizeof(int) * nq) == 0;
  }
};

// Qubit a primitive needs on a register bit, or -1 (diagonal gates and CNOT
// controls work from any physical bit).
int register_need(const Prim& p) {
  switch (p.kind) {
    case P_RX:
    case P_RY:
      return p.q0;
    case P_CNOT:
      return p.q1;
    default:
      return -1;
  }
}

bool two_qubit(const Prim& p) { return p.kind == P_CNOT || p.kind == P_CZ; }

// next_need[i * nq + q]: first index >= i of `seq` that needs q on a register.
std::vector<int> next_need_table(const std::vector<Prim>& seq, int nq) {
  const int G = (int)seq.size();
  std::vector<int> t((size_t)(G + 1) * nq, INT_MAX);
  for (int i = G - 1; i >= 0; --i) {
    for (int q = 0; q < nq; ++q) t[(size_t)i * nq + q] = t[(size_t)(i + 1) * nq + q];
    const int need = register_need(seq[i]);
    if (need >= 0) t[(size_t)i * nq + need] = i;
  }
  return t;
}

// Exchange tables.  The LDS slot of an amplitude is a GF(2)-linear function
// lam(x) of its tile position, chosen so that the lanes of a 32-lane group hit
// 32 distinct banks both when writing in the old layout and when reading in the
// new one.  With A the qubits on the old layout's first lane bits and B those
// of the new layout: the qubit of A at lane i gets slot bit i; each qubit of
// B \ A shares the slot bit of a distinct qubit of A \ B (so the slot bits of B
// are independent too); every qubit outside A also gets one high bit of its
// own, which keeps lam invertible (triangular).
int emit_exchange(const Mapping& a, const Mapping& b, int k, int R, std::vector<uint32_t>& cols) {
  const int t = k - R;
  const int lb = std::min(kBankBits, t);
  uint32_t lam[kMaxQubits];
  bool in_a[kMaxQubits], in_b[kMaxQubits];
  std::memset(lam, 0, sizeof(lam));
  std::memset(in_a, 0, sizeof(in_a));
  std::memset(in_b, 0, sizeof(in_b));
  for (int i = 0; i < lb; ++i) {
    in_a[a.p2q[R + i]] = true;
    in_b[b.p2q[R + i]] = true;
  }
  std::vector<int> a_only_bit, b_only;
  for (int i = 0; i < lb; ++i) {
    const int qa = a.p2q[R + i];
    lam[qa] |= 1u << i;
    if (!in_b[qa]) a_only_bit.push_back(i);
  }
  for (int i = 0; i < lb; ++i) {
    const int qb = b.p2q[R + i];
    if (!in_a[qb]) b_only.push_back(qb);
  }
  for (size_t j = 0; j < b_only.size(); ++j) lam[b_only[j]] |= 1u << a_only_bit[j];
  int nb = lb;
  for (int p = 0; p < k; ++p) {
    const int q = a.p2q[p];
    if (!in_a[q]) lam[q] |= 1u << nb++;
  }
  const int off = (int)cols.size();
  for (int p = 0; p < k; ++p) cols.push_back(lam[a.p2q[p]]);
  for (int p = 0; p < k; ++p) cols.push_back(lam[b.p2q[p]]);
  // then where each physical bit's qubit goes (the generated kernels do
  // exchanges that only swap register bits with lane bits without LDS)
  for (int p = 0; p < k; ++p) cols.push_back((uint32_t)b.q2p[a.p2q[p]]);
  return off;
}

void emit(std::vector<uint32_t>& out, uint32_t op, int a, int b, int slot, uint32_t arg) {
  out.push_back(ins_word0(op, (uint32_t)a, (uint32_t)b, slot));
  out.push_back(arg);
}

// A list schedule of `seq` that holds back RZs with variable angles until no
// other gate is ready, then emits every ready one and those they make ready,
// so that they come in runs over many qubits (the
// generated kernels with 8 or more amplitudes per thread apply such a run as
// one diagonal: a Rot layer becomes the RZs of every qubit, the RYs, then the
// other RZs).  Each line keeps its order of gates; among ready gates the one
// earlier in `seq` goes first, so the gates that need a register bit keep
// their order.
std::vector<Prim> lazy_diagonals(const std::vector<Prim>& seq, const Plan& plan) {
  const int n = (int)seq.size();
  std::vector<int> npred(n, 0);
  std::vector<std::vector<int>> succ(n);
  int last[kMaxQubits];
  for (int q = 0; q < kMaxQubits; ++q) last[q] = -1;
  for (int i = 0; i < n; ++i) {
    const int lines[2] = {seq[i].q0, two_qubit(seq[i]) ? seq[i].q1 : -1};
    for (int q : lines) {
      if (q < 0) continue;
      if (last[q] >= 0) {
        succ[last[q]].push_back(i);
        ++npred[i];
      }
      last[q] = i;
    }
  }
  auto held = [&](int i) {
    return seq[i].kind == P_RZ && seq[i].occ >= 0 && plan.occ_src[seq[i].occ] != VQC_SRC_CONST;
  };
  std::set<int> other, rz;
  for (int i = 0; i < n; ++i)
    if (!npred[i]) (held(i) ? rz : other).insert(i);
  std::vector<Prim> out;
  out.reserve(n);
  auto take = [&](int i) {
    out.push_back(seq[i]);
    for (int s : succ[i])
      if (--npred[s] == 0) (held(s) ? rz : other).insert(s);
  };
  while ((int)out.size() < n) {
    if (!other.empty()) {
      const int i = *other.begin();
      other.erase(other.begin());
      take(i);
    } else {  // every ready RZ, and those they make ready (a qubit's next RZ)
      while (!rz.empty()) {
        const int i = *rz.begin();
        rz.erase(rz.begin());
        take(i);
      }
    }
  }
  return out;
}

// One register-level sweep over `seq` (already in execution order) starting
// from mapping `m` (updated to the end mapping).  slot_of(occ) gives the
// gradient accumulator written into rotation instructions.
// `lanes` > 0: RX / RY and CNOT targets may also act on the first `lanes`
// thread bits (lane bits of the sample; generated kernels only).
template <typename SlotFn>
int plan_sweep(const std::vector<Prim>& seq, int nq, int k, int R, Mapping& m,
               std::vector<uint32_t>& out, std::vector<uint32_t>& cols, int& exchanges,
               SlotFn slot_of, std::string& msg, int lanes = 0) {
  const std::vector<int> nn = next_need_table(seq, nq);
  for (size_t i = 0; i < seq.size(); ++i) {
    const Prim& pr = seq[i];
    const int need = register_need(pr);
    if (need >= 0 && m.q2p[need] >= k) {
      msg = "internal: register-bit gate on a global qubit";
      return VQC_ERR_UNSUPPORTED;
    }
    if (need >= 0 && m.q2p[need] >= R + lanes) {
      // Belady: the register bits get the R local qubits needed soonest.  A
      // qubit on a lane bit that takes gates needs no register.
      std::vector<int> qs;
      for (int p = 0; p < k; ++p) qs.push_back(m.p2q[p]);
      const int* nrow = &nn[i * (size_t)nq];
      auto row_of = [&](int q) {
        const int p = m.q2p[q];
        return (p >= R && p < R + lanes) ? INT_MAX : nrow[q];
      };
      std::stable_sort(qs.begin(), qs.end(), [&](int x, int y) {
        const int rx_need = row_of(x), ry_need = row_of(y);
        if (rx_need != ry_need) return rx_need < ry_need;
        const bool rx = m.q2p[x] < R, ry = m.q2p[y] < R;
        if (rx != ry) return rx;  // keep residents on ties
        return x < y;
      });
      bool chosen[kMaxQubits] = {false};
      for (int r = 0; r < R; ++r) chosen[qs[r]] = true;
      std::vector<int> incoming, outgoing;
      for (int r = 0; r < R; ++r)
        if (!chosen[m.p2q[r]]) outgoing.push_back(r);
      for (int r = 0; r < R; ++r)
        if (m.q2p[qs[r]] >= R) incoming.push_back(qs[r]);
      Mapping nm = m;
      for (size_t j = 0; j < incoming.size(); ++j) {
        const int qin = incoming[j];
        const int pin = m.q2p[qin];
        const int pout = outgoing[j];
        const int qout = m.p2q[pout];
        nm.p2q[pout] = qin;
        nm.q2p[qin] = pout;
        nm.p2q[pin] = qout;
        nm.q2p[qout] = pin;
      }
      emit(out, OP_EXCHANGE, 0, 0, -1, (uint32_t)emit_exchange(m, nm, k, R, cols));
      ++exchanges;
      m = nm;
    }
    switch (pr.kind) {
      case P_RX: emit(out, OP_RX, m.q2p[pr.q0], 0, slot_of(pr.occ), (uint32_t)pr.occ); break;
      case P_RY: emit(out, OP_RY, m.q2p[pr.q0], 0, slot_of(pr.occ), (uint32_t)pr.occ); break;
      case P_RZ: emit(out, OP_RZ, m.q2p[pr.q0], 0, slot_of(pr.occ), (uint32_t)pr.occ); break;
      case P_CNOT: emit(out, OP_CNOT, m.q2p[pr.q0], m.q2p[pr.q1], -1, 0); break;
      case P_CZ: emit(out, OP_CZ, m.q2p[pr.q0], m.q2p[pr.q1], -1, 0); break;
      default: msg = "internal: unknown primitive"; return VQC_ERR_UNSUPPORTED;
    }
  }
  return 0;
}

int append_map(const Mapping& m, std::vector<uint8_t>& maps) {
  const int off = (int)maps.size();
  for (int q = 0; q < m.nq; ++q) maps.push_back((uint8_t)m.q2p[q]);
  return off;
}

// ------------------------------------------------------------ streaming passes
// A pass holds k local qubits of one sample per workgroup; the other ng global
// qubits are fixed by the workgroup's tile index.  Between two passes the state
// sits in HBM in a memory layout of its own: a permutation of the qubits over
// the address bits, chosen so that the qubits local in both the writing and
// the reading pass take the lowest address bits.  Any qubit may then be global
// in a pass (the tile I/O of both passes stays in runs of consecutive
// addresses), so a pass takes the global set that lets it run the most gates.

// A pass before its sweep is planned: its global qubits and the gates it runs.
struct StreamGroup {
  uint32_t glob = 0;
  std::vector<Prim> prims;
};

uint32_t lines_of(const Prim& p) {
  return (1u << p.q0) | (two_qubit(p) ? 1u << p.q1 : 0u);
}

// The gates of `seq` not yet done that one pass with global set `glob` runs:
// in circuit order, every gate whose lines no earlier waiting gate blocks and
// whose register qubit is local.  Returns their count; `took` gets them.
int pass_gates(const std::vector<Prim>& seq, const std::vector<char>& done, uint32_t glob,
               uint32_t all, std::vector<int>* took) {
  uint32_t blocked = 0;
  int count = 0;
  for (size_t i = 0; i < seq.size() && blocked != all; ++i) {
    if (done[i]) continue;
    const Prim& p = seq[i];
    const uint32_t lines = lines_of(p);
    const int need = register_need(p);
    if (!(blocked & lines) && (need < 0 || !((glob >> need) & 1u))) {
      ++count;
      if (took) took->push_back((int)i);
    } else {
      blocked |= lines;
    }
  }
  return count;
}

uint64_t binomial(int n, int r) {
  uint64_t v = 1;
  for (int i = 1; i <= r; ++i) v = v * (uint64_t)(n - r + i) / (uint64_t)i;
  return v;
}

constexpr uint64_t kMaxGlobalCandidates = 20000;

// Pass partition.  Each pass takes, among all sets of ng qubits, the one that
// lets it run the most gates; ties go to the set whose qubits are needed on a
// register latest.  With more than kMaxGlobalCandidates sets, the ng qubits
// needed latest.
int partition_stream(const std::vector<Prim>& seq, int nq, int ng,
                     std::vector<StreamGroup>& groups, std::string& msg) {
  const uint32_t all = nq >= 32 ? ~0u : (1u << nq) - 1u;
  std::vector<char> done(seq.size(), 0);
  size_t remaining = seq.size();
  const bool search = binomial(nq, ng) <= kMaxGlobalCandidates;
  do {
    // rank of each qubit's first pending register need (never needed: last)
    int rank[kMaxQubits];
    for (int q = 0; q < nq; ++q) rank[q] = INT_MAX;
    int r = 0;
    for (size_t i = 0; i < seq.size(); ++i) {
      if (done[i]) continue;
      const int q = register_need(seq[i]);
      if (q >= 0 && rank[q] == INT_MAX) rank[q] = r++;
    }
    for (int q = 0; q < nq; ++q)
      if (rank[q] == INT_MAX) rank[q] = r++;
    uint32_t best = 0;
    if (ng > 0) {
      // the ng qubits needed latest
      std::vector<int> order(nq);
      for (int q = 0; q < nq; ++q) order[rank[q]] = q;
      for (int j = 0; j < ng; ++j) best |= 1u << order[nq - 1 - j];
      if (search) {
        int best_count = -1;
        long best_tie = -1;
        // every ng-subset of the nq qubits (Gosper's enumeration of masks)
        for (uint32_t g = (1u << ng) - 1u; g <= all && g != 0;) {
          const int c = pass_gates(seq, done, g, all, nullptr);
          long tie = 0;
          for (int q = 0; q < nq; ++q)
            if ((g >> q) & 1u) tie += rank[q];
          if (c > best_count || (c == best_count && tie > best_tie)) {
            best_count = c;
            best_tie = tie;
            best = g;
          }
          const uint32_t lo = g & (0u - g), hi = g + lo;
          if (hi == 0) break;
          g = (((hi ^ g) >> 2) / lo) | hi;
        }
      }
    }
    std::vector<int> took;
    pass_gates(seq, done, best, all, &took);
    if (took.empty() && remaining > 0) {
      msg = "internal: streaming pass made no progress";
      return VQC_ERR_UNSUPPORTED;
    }
    StreamGroup grp;
    grp.glob = best;
    for (int i : took) {
      grp.prims.push_back(seq[i]);
      done[i] = 1;
    }
    remaining -= took.size();
    groups.push_back(std::move(grp));
  } while (remaining > 0);
  return 0;
}

// Memory layout at the boundary between a pass that writes (global set
// wglob) and one that reads (rglob): the qubits local in both come first
// (ascending), then the others (ascending).  pos[q] = address bit of qubit q.
void boundary_layout(uint32_t wglob, uint32_t rglob, int nq, int* pos) {
  int b = 0;
  for (int q = 0; q < nq; ++q)
    if (!((wglob >> q) & 1u) && !((rglob >> q) & 1u)) pos[q] = b++;
  for (int q = 0; q < nq; ++q)
    if (((wglob >> q) & 1u) || ((rglob >> q) & 1u)) pos[q] = b++;
}

void identity_layout(int nq, int* pos) {
  for (int q = 0; q < nq; ++q) pos[q] = q;
}

// Tile I/O mapping of a pass for memory layout `pos`: the local qubits ordered
// by address bit are the tile ranks; ranks 0..k-R-1 sit on the thread bits and
// the top R on the register bits, so consecutive lanes touch consecutive
// addresses.  Global qubits, ascending, take the tile index bits.
Mapping io_mapping(uint32_t glob, const int* pos, int k, int R, int nq) {
  Mapping m;
  m.k = k;
  m.nq = nq;
  for (int q = 0; q < kMaxQubits; ++q) m.q2p[q] = -1;
  std::vector<int> local;
  for (int q = 0; q < nq; ++q)
    if (!((glob >> q) & 1u)) local.push_back(q);
  std::sort(local.begin(), local.end(), [&](int x, int y) { return pos[x] < pos[y]; });
  const int nt = k - R;
  for (int r = 0; r < k; ++r) {
    const int p = r < nt ? R + r : r - nt;
    m.p2q[p] = local[r];
    m.q2p[local[r]] = p;
  }
  int j = 0;
  for (int q = 0; q < nq; ++q)
    if ((glob >> q) & 1u) m.q2p[q] = k + j++;
  return m;
}

// The k + ng address columns of a tile under mapping m and layout pos: one per
// tile rank (thread bits first, then register bits), then one per global bit.
// Addresses are the XOR of the columns of the set bits; with `col` a qubit's
// column is col[pos[q]] instead of a single bit (a GF(2) map of the index).
void push_io(const Mapping& m, const int* pos, int k, int R, std::vector<uint32_t>& cols,
             const uint32_t* col = nullptr) {
  const int nt = k - R;
  auto c = [&](int q) { return col ? col[pos[q]] : 1u << pos[q]; };
  for (int r = 0; r < k; ++r) {
    const int p = r < nt ? R + r : r - nt;
    cols.push_back(c(m.p2q[p]));
  }
  std::vector<uint32_t> g(m.nq - k, 0u);
  for (int q = 0; q < m.nq; ++q)
    if (m.q2p[q] >= k) g[m.q2p[q] - k] = c(q);
  cols.insert(cols.end(), g.begin(), g.end());
}

// True if the n columns at cols[off] are distinct single bits: a tile's loads
// and stores add a lane's address bits to a register's (streaming kernel).
bool one_hot_columns(const std::vector<uint32_t>& cols, int off, int n) {
  uint32_t seen = 0;
  for (int i = 0; i < n; ++i) {
    const uint32_t c = cols[off + i];
    if (c == 0 || (c & (c - 1)) || (seen & c)) return false;
    seen |= c;
  }
  return true;
}

// Plans the sweeps of the passes `groups` (one direction): each starts in the
// tile I/O mapping of its input layout, runs its gates, and ends in the I/O
// mapping of its output layout (no closing exchange when it stores nothing).
// in_pos / out_pos: the layout each pass reads / writes.
int plan_stream(Plan& plan, const std::vector<StreamGroup>& groups,
                const std::vector<std::vector<int>>& in_pos,
                const std::vector<std::vector<int>>& out_pos, bool bwd, int R,
                std::vector<uint32_t>& out, std::vector<PassPlan>& passes, int& exchanges,
                std::string& msg) {
  const int nq = plan.nq, k = plan.k;
  int ident[kMaxQubits];
  identity_layout(nq, ident);
  for (size_t i = 0; i < groups.size(); ++i) {
    const StreamGroup& grp = groups[i];
    const bool last = i + 1 == groups.size();
    const Mapping io_in = io_mapping(grp.glob, in_pos[i].data(), k, R, nq);
    const Mapping io_out = io_mapping(grp.glob, out_pos[i].data(), k, R, nq);
    Mapping m = io_in;
    PassPlan pp;
    pp.ins_off = (int)out.size() / 2;
    pp.start_off = append_map(io_in, plan.maps);
    std::map<int, int> local_slot;
    std::vector<int32_t> slots;
    auto slot_of = [&](int occ) -> int {
      const int s = plan.occ_slot[occ];
      if (s < 0) return -1;
      auto it = local_slot.find(s);
      if (it != local_slot.end()) return it->second;
      const int id = (int)slots.size();
      local_slot[s] = id;
      slots.push_back(s);
      return id;
    };
    const std::vector<Prim> seq = R >= 3 ? lazy_diagonals(grp.prims, plan) : grp.prims;
    int rc = plan_sweep(seq, nq, k, R, m, out, plan.cols, exchanges, slot_of, msg);
    if (rc < 0) return rc;
    const bool stores = !(bwd && last);  // the adjoint's last pass ends at psi_0
    if (stores && !(m == io_out)) {
      emit(out, OP_EXCHANGE, 0, 0, -1, (uint32_t)emit_exchange(m, io_out, k, R, plan.cols));
      ++exchanges;
      m = io_out;
    }
    pp.end_off = append_map(m, plan.maps);
    pp.n_ins = (int)out.size() / 2 - pp.ins_off;
    pp.io_off = (int)plan.cols.size();
    push_io(io_in, in_pos[i].data(), k, R, plan.cols);
    pp.io_out_off = (int)plan.cols.size();
    push_io(m, stores ? out_pos[i].data() : ident, k, R, plan.cols);
    pp.io_lin_off = (int)plan.cols.size();
    push_io(io_in, ident, k, R, plan.cols);
    pp.io_lout_off = (int)plan.cols.size();
    push_io(m, ident, k, R, plan.cols, plan.pcol.empty() ? nullptr : plan.pcol.data());
    if (!one_hot_columns(plan.cols, pp.io_off, nq) || !one_hot_columns(plan.cols, pp.io_out_off, nq) ||
        !one_hot_columns(plan.cols, pp.io_lin_off, nq)) {
      msg = "internal: tile address columns are not distinct bits";
      return VQC_ERR_UNSUPPORTED;
    }
    pp.slots_off = (int)plan.pslots.size();
    pp.n_slots = (int)slots.size();
    plan.pslots.insert(plan.pslots.end(), slots.begin(), slots.end());
    plan.max_pass_slots = std::max(plan.max_pass_slots, pp.n_slots);
    if (i == 0) pp.flags |= bwd ? PF_MAKE_LAMBDA : PF_INIT;
    if (last) pp.flags |= bwd ? PF_LAST_ADJ : PF_ZPART;
    passes.push_back(pp);
  }
  return 0;
}

// Both directions of the streaming path.  The forward is partitioned into
// passes; the adjoint runs the same passes in reverse order, each over its
// forward pass's gates reversed, so that it reads the state that forward pass
// saved (a training forward keeps every pass's output) instead of rewriting
// psi: an adjoint pass reads psi and lambda and writes only lambda.  The
// forward's first pass reads (Psi_0) in logical order; the mirror of pass i
// reads in the layout pass i wrote and writes in the layout pass i read.
int plan_stream_both(Plan& plan, std::string& msg) {
  const int nq = plan.nq;
  std::vector<StreamGroup> fg;
  int rc = partition_stream(plan.prims, nq, plan.ng, fg, msg);
  if (rc < 0) return rc;
  const size_t nf = fg.size();
  std::vector<StreamGroup> bg(nf);
  for (size_t j = 0; j < nf; ++j) {
    const StreamGroup& f = fg[nf - 1 - j];
    bg[j].glob = f.glob;
    bg[j].prims.assign(f.prims.rbegin(), f.prims.rend());
  }
  std::vector<std::vector<int>> fin(nf, std::vector<int>(nq)), fout(nf, std::vector<int>(nq));
  std::vector<std::vector<int>> bin(nf, std::vector<int>(nq)), bout(nf, std::vector<int>(nq));
  identity_layout(nq, fin[0].data());
  for (size_t i = 0; i < nf; ++i) {
    // the last output is read by its own mirror: same local qubits on both sides
    const uint32_t next = i + 1 < nf ? fg[i + 1].glob : fg[i].glob;
    boundary_layout(fg[i].glob, next, nq, fout[i].data());
    if (i + 1 < nf) fin[i + 1] = fout[i];
  }
  for (size_t j = 0; j < nf; ++j) {
    bin[j] = fout[nf - 1 - j];
    if (j + 1 < nf) bout[j] = fin[nf - 1 - j];
    else identity_layout(nq, bout[j].data());  // the last adjoint pass stores nothing
  }
  rc = plan_stream(plan, fg, fin, fout, false, plan.Rf, plan.fwd, plan.fpass, plan.fwd_exchanges,
                   msg);
  if (rc < 0) return rc;
  return plan_stream(plan, bg, bin, bout, true, plan.Rb, plan.bwd, plan.bpass,
                     plan.bwd_exchanges, msg);
}

// ------------------------------------------------------------- lowering
// Every gate of the static set becomes primitives the kernels run: Pauli
// rotations R_P(t) = exp(-i t P / 2) on one qubit, CNOT and CZ.  The products
// equal the gate up to a global phase (which no output depends on); each is a
// standard identity: H ~ RY(pi/2) RZ(pi); S, T, P ~ RZ; SX ~ RX(pi/2);
// U3(t, p, l) ~ RZ(p) RY(t) RZ(l); controlled rotations split into half-angle
// rotations around two CNOTs; R_ZZ is a CNOT-conjugated RZ and R_XX, R_YY add
// basis changes; CY, CH conjugate CNOT / CZ by target rotations; SWAP is three
// CNOTs; CCX is the six-CNOT Toffoli circuit of Nielsen and Chuang (Fig. 4.9);
// CSWAP is a Toffoli between two CNOTs.

struct GateShape {
  int wires, angles;
};

GateShape gate_shape(int kind) {
  switch (kind) {
    case VQC_RX: case VQC_RY: case VQC_RZ: case VQC_P: return {1, 1};
    case VQC_ROT: case VQC_U3: return {1, 3};
    case VQC_U2: return {1, 2};
    case VQC_CNOT: case VQC_CZ: case VQC_CY: case VQC_CH: case VQC_SWAP: return {2, 0};
    case VQC_CRX: case VQC_CRY: case VQC_CRZ: case VQC_CP: case VQC_RXX: case VQC_RYY:
    case VQC_RZZ: return {2, 1};
    case VQC_CCX: case VQC_CSWAP: return {3, 0};
    default: return {1, 0};  // ID and the fixed one-qubit gates
  }
}

constexpr double kPi = 3.14159265358979323846;

// (cos, sin)(th / 2) of a constant rotation in float.  The nearest floats of
// common angles all shrink the norm the same way (cos^2 + sin^2 - 1 is about
// -3e-8 at 45 and 22.5 degrees), so that a circuit with hundreds of such gates
// loses 1e-5 of its norm.  Among the pairs within one float step of the
// nearest ones this takes the pair whose norm error brings the running sum of
// the circuit's errors (drift) closest to zero (ties: the nearer pair), which
// keeps the product of the constant gates' norms within one step's error of 1.
void constant_pair(double th, double& drift, float& c, float& s) {
  const double cd = std::cos(0.5 * th), sd = std::sin(0.5 * th);
  const float c0 = (float)cd, s0 = (float)sd;
  const float cs[3] = {std::nextafter(c0, -2.f), c0, std::nextafter(c0, 2.f)};
  const float ss[3] = {std::nextafter(s0, -2.f), s0, std::nextafter(s0, 2.f)};
  double best = -1.0, best_d = 0.0, best_e = 0.0;
  for (float cc : cs)
    for (float sc : ss) {
      const double e = (double)cc * cc + (double)sc * sc - 1.0;
      const double score = std::fabs(drift + e), d = std::fabs(cc - cd) + std::fabs(sc - sd);
      if (best < 0.0 || score < best || (score == best && d < best_d)) {
        best = score;
        best_d = d;
        best_e = e;
        c = cc;
        s = sc;
      }
    }
  drift += best_e;
}

// Emits the primitives of one (validated) gate into plan.prims, with one
// angle occurrence per rotation: m * (the gate's angle slot s) + a, or the
// constant a when s < 0.
class Lowering {
 public:
  Lowering(const HostOp& o, Plan& p) : o_(o), p_(p) {}

  void rot(int kind, int q, int s, double m = 1.0, double a = 0.0) {
    const int occ = (int)p_.occ_src.size();
    const int src = s < 0 ? VQC_SRC_CONST : o_.src[s];
    if (src == VQC_SRC_CONST) {
      // constant gates are cached at compile time (Algorithm 1, compile phase)
      const double th = s < 0 ? a : m * (double)o_.val[s] + a;
      p_.occ_src.push_back(VQC_SRC_CONST);
      p_.occ_idx.push_back(0);
      p_.occ_slot.push_back(-1);
      float c = 0.f, sn = 0.f;
      constant_pair(th, p_.const_drift, c, sn);
      p_.occ_cs.push_back(c);
      p_.occ_cs.push_back(sn);
      p_.occ_ma.push_back(1.f);
      p_.occ_ma.push_back(0.f);
    } else {
      const int idx = o_.idx[s];
      const float mul = (float)(m * (double)o_.mul[s]);
      const float add = (float)(m * (double)o_.val[s] + a);
      p_.occ_src.push_back(src);
      p_.occ_idx.push_back(idx);
      p_.occ_slot.push_back(src == VQC_SRC_PARAM ? idx : p_.P + idx);
      p_.occ_cs.push_back(0.f);
      p_.occ_cs.push_back(0.f);
      p_.occ_ma.push_back(mul);
      p_.occ_ma.push_back(add);
      if (mul != 1.f || add != 0.f) p_.affine = true;
    }
    p_.prims.push_back({kind, q, -1, occ});
  }
  void cnot(int c, int t) { p_.prims.push_back({P_CNOT, c, t, -1}); }
  void cz(int a, int b) { p_.prims.push_back({P_CZ, a, b, -1}); }
  void c_rz(int q, double a) { rot(P_RZ, q, -1, 1.0, a); }
  void c_ry(int q, double a) { rot(P_RY, q, -1, 1.0, a); }
  void c_rx(int q, double a) { rot(P_RX, q, -1, 1.0, a); }
  void h(int q) {
    c_rz(q, kPi);
    c_ry(q, kPi / 2);
  }
  void toffoli(int a, int b, int c) {
    h(c);
    cnot(b, c);
    c_rz(c, -kPi / 4);
    cnot(a, c);
    c_rz(c, kPi / 4);
    cnot(b, c);
    c_rz(c, -kPi / 4);
    cnot(a, c);
    c_rz(b, kPi / 4);
    c_rz(c, kPi / 4);
    h(c);
    cnot(a, b);
    c_rz(a, kPi / 4);
    c_rz(b, -kPi / 4);
    cnot(a, b);
  }

 private:
  const HostOp& o_;
  Plan& p_;
};

void lower_gate(const HostOp& o, Plan& plan) {
  Lowering L(o, plan);
  const int a = o.w[0], b = o.w[1], c = o.w[2];
  switch (o.kind) {
    case VQC_RX: L.rot(P_RX, a, 0); break;
    case VQC_RY: L.rot(P_RY, a, 0); break;
    case VQC_RZ: L.rot(P_RZ, a, 0); break;
    case VQC_ROT:  // RZ(omega) RY(theta) RZ(phi): phi first
      L.rot(P_RZ, a, 0);
      L.rot(P_RY, a, 1);
      L.rot(P_RZ, a, 2);
      break;
    case VQC_CNOT: L.cnot(a, b); break;
    case VQC_CZ: L.cz(a, b); break;
    case VQC_ID: break;
    case VQC_X: L.c_rx(a, kPi); break;
    case VQC_Y: L.c_ry(a, kPi); break;
    case VQC_Z: L.c_rz(a, kPi); break;
    case VQC_H: L.h(a); break;
    case VQC_S: L.c_rz(a, kPi / 2); break;
    case VQC_SDG: L.c_rz(a, -kPi / 2); break;
    case VQC_T: L.c_rz(a, kPi / 4); break;
    case VQC_TDG: L.c_rz(a, -kPi / 4); break;
    case VQC_SX: L.c_rx(a, kPi / 2); break;
    case VQC_SXDG: L.c_rx(a, -kPi / 2); break;
    case VQC_P: L.rot(P_RZ, a, 0); break;
    case VQC_U2:  // U3(pi/2, phi, lambda)
      L.rot(P_RZ, a, 1);
      L.c_ry(a, kPi / 2);
      L.rot(P_RZ, a, 0);
      break;
    case VQC_U3:  // RZ(phi) RY(theta) RZ(lambda): lambda first
      L.rot(P_RZ, a, 2);
      L.rot(P_RY, a, 0);
      L.rot(P_RZ, a, 1);
      break;
    case VQC_CY:
      L.c_rz(b, -kPi / 2);
      L.cnot(a, b);
      L.c_rz(b, kPi / 2);
      break;
    case VQC_CH:
      L.c_ry(b, -kPi / 4);
      L.cz(a, b);
      L.c_ry(b, kPi / 4);
      break;
    case VQC_SWAP:
      L.cnot(a, b);
      L.cnot(b, a);
      L.cnot(a, b);
      break;
    case VQC_CRX:
      L.c_rz(b, kPi / 2);
      L.rot(P_RY, b, 0, 0.5);
      L.cnot(a, b);
      L.rot(P_RY, b, 0, -0.5);
      L.cnot(a, b);
      L.c_rz(b, -kPi / 2);
      break;
    case VQC_CRY:
    case VQC_CRZ: {
      const int pk = o.kind == VQC_CRY ? P_RY : P_RZ;
      L.rot(pk, b, 0, 0.5);
      L.cnot(a, b);
      L.rot(pk, b, 0, -0.5);
      L.cnot(a, b);
      break;
    }
    case VQC_CP:
      L.rot(P_RZ, a, 0, 0.5);
      L.rot(P_RZ, b, 0, 0.5);
      L.cnot(a, b);
      L.rot(P_RZ, b, 0, -0.5);
      L.cnot(a, b);
      break;
    case VQC_RXX:
    case VQC_RYY:
    case VQC_RZZ: {
      // basis change B with B Z B^dagger = X (RY(pi/2)) or Y (RX(-pi/2))
      const bool xx = o.kind == VQC_RXX, yy = o.kind == VQC_RYY;
      if (xx) { L.c_ry(a, -kPi / 2); L.c_ry(b, -kPi / 2); }
      if (yy) { L.c_rx(a, kPi / 2); L.c_rx(b, kPi / 2); }
      L.cnot(a, b);
      L.rot(P_RZ, b, 0);
      L.cnot(a, b);
      if (xx) { L.c_ry(a, kPi / 2); L.c_ry(b, kPi / 2); }
      if (yy) { L.c_rx(a, -kPi / 2); L.c_rx(b, -kPi / 2); }
      break;
    }
    case VQC_CCX: L.toffoli(a, b, c); break;
    case VQC_CSWAP:
      L.cnot(c, b);
      L.toffoli(a, b, c);
      L.cnot(c, b);
      break;
    default: break;
  }
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

// Measurement of the trailing entanglers.  A CNOT or CZ none of whose qubits
// carries a later rotation can move to the end of the circuit (everything after
// it on its lines is such a gate too), and the entanglers there need not run:
// with T their product, <Z_j> of the final state is <psi| T^dag Z_j T |psi> for
// the state psi before them, and T^dag Z_j T is a Z-string (CNOT(c, t) takes Z_t
// to Z_c Z_t, CZ leaves Z-strings alone); the probability of basis state A x
// after them is that of x before them, A the GF(2) map of the CNOTs.  The
// adjoint starts from lambda = (sum_j g_j T^dag Z_j T) psi.  (The tangent
// form's frame rows still propagate through the tail: they describe the final
// state.)
//
// Diagonal gates (RZ, CZ) that commute with every gate kept after them are
// dropped: moved to the end they act on a state whose every output is
// diagonal in the computational basis (<Z>-strings and probabilities), so
// neither the outputs nor any other gate's gradient change, and their own
// gradients are zero (Im <psi| H |psi> = 0 for the diagonal Hermitian H the
// adjoint pairs them with).  A diagonal gate commutes with diagonal gates and
// CNOT controls; RX, RY and CNOT targets on its qubits block it.  One
// backward scan decides both, each gate against the final form of the gates
// after it (kept ones in place, folded ones at the end, dropped ones gone).
void fold_trailing_entanglers(Plan& plan) {
  // 0 keep, 1 tail (folded into the measurement), 2 dropped
  std::vector<char> tail(plan.prims.size(), 0);
  uint32_t blocked = 0;  // lines of a later kept gate (the fold rule)
  uint32_t noncomm = 0;  // qubits of a later kept RX, RY or CNOT target (the drop rule)
  bool any = false;
  for (size_t i = plan.prims.size(); i-- > 0;) {
    const Prim& g = plan.prims[i];
    const uint32_t lines = lines_of(g);
    const bool diagonal = g.kind == P_RZ || g.kind == P_CZ;
    if (diagonal && !(noncomm & lines)) {
      tail[i] = 2;
      any = true;
    } else if (g.kind == P_CNOT && !(blocked & lines)) {
      tail[i] = 1;
      any = true;
    } else {
      blocked |= lines;
      if (g.kind == P_RX || g.kind == P_RY) noncomm |= lines;
      if (g.kind == P_CNOT) noncomm |= 1u << g.q1;
    }
  }
  if (!any) return;
  std::vector<Prim> body;
  for (size_t i = 0; i < plan.prims.size(); ++i) {
    if (tail[i] == 0) body.push_back(plan.prims[i]);
    else if (tail[i] == 1) plan.tail.push_back(plan.prims[i]);
  }
  plan.prims.swap(body);
  if (plan.tail.empty()) return;
  plan.zmask.assign(plan.n, 0u);
  for (int j = 0; j < plan.n; ++j) {
    uint32_t m = 1u << j;
    for (size_t i = plan.tail.size(); i-- > 0;) {
      const Prim& g = plan.tail[i];
      if (g.kind == P_CNOT && ((m >> g.q1) & 1u)) m ^= 1u << g.q0;
    }
    plan.zmask[j] = m;
  }
  plan.pcol.assign(plan.n, 0u);
  for (size_t q = 0; q < plan.pcol.size(); ++q) {
    uint32_t v = 1u << q;
    for (const Prim& g : plan.tail)
      if (g.kind == P_CNOT && ((v >> g.q0) & 1u)) v ^= 1u << g.q1;
    plan.pcol[q] = v;
  }
}

// Each qubit's head (the rotations on it before the first entangler on it).
void find_heads(Plan& plan) {
  plan.head.assign(plan.n, {});
  uint32_t blocked = 0;
  for (const Prim& g : plan.prims) {
    const uint32_t lines = lines_of(g);
    const bool rot = g.kind == P_RX || g.kind == P_RY || g.kind == P_RZ;
    if (rot && g.occ >= 0 && !(blocked & lines))
      plan.head[g.q0].push_back(g);
    else
      blocked |= lines;
  }
}

// LDS of the streaming passes: exchange buffer | angle table | gradient
// accumulators [slot][group] of the adjoint.
void stream_lds(Plan& plan) {
  const size_t xbuf = ((size_t)1 << plan.k) * 8;
  plan.lds_tab = xbuf;
  const size_t tab = align_up(plan.occ_src.size() * 8, 16);
  plan.lds_acc = xbuf + tab;
  const size_t groups_bwd = ((size_t)1 << (plan.k - plan.Rb)) / 64;
  const size_t acc = align_up((size_t)plan.max_pass_slots * groups_bwd * 4, 16);
  plan.lds_fwd = xbuf + tab;
  plan.lds_bwd = xbuf + tab + acc;
}

int build_plan(const std::vector<HostOp>& ops, int n, int P, int F, int path, int reg_bits,
               Plan& plan, std::string& msg, bool lane_gates, int tile_qubits) {
  if (n < 1 || n > kMaxQubits) {
    msg = "n_qubits must be in [1, " + std::to_string(kMaxQubits) + "]";
    return n < 1 ? VQC_ERR_INVALID_ARG : VQC_ERR_TOO_LARGE;
  }
  if (P < 0 || F < 0) {
    msg = "n_params and n_inputs must be >= 0";
    return VQC_ERR_INVALID_ARG;
  }
  plan = Plan();
  plan.n = n;
  plan.P = P;
  plan.F = F;
  plan.n_ops = (int)ops.size();
  // validation and lowering (Sec. 3 "Static Circuit Scope": gate identity and
  // wiring are fixed here; only angles vary at run time)
  for (size_t k = 0; k < ops.size(); ++k) {
    const HostOp& o = ops[k];
    const std::string at = "op " + std::to_string(k) + ": ";
    if (o.kind < 0 || o.kind >= kNumGateKinds) {
      msg = at + "unknown kind " + std::to_string(o.kind);
      return VQC_ERR_INVALID_ARG;
    }
    const GateShape sh = gate_shape(o.kind);
    for (int i = 0; i < sh.wires; ++i) {
      if (o.w[i] < 0 || o.w[i] >= n) {
        msg = at + "wire " + std::to_string(o.w[i]) + " out of range";
        return VQC_ERR_INVALID_ARG;
      }
      for (int j = 0; j < i; ++j)
        if (o.w[j] == o.w[i]) {
          msg = at + "a wire appears twice in one gate";
          return VQC_ERR_INVALID_ARG;
        }
    }
    for (int s = 0; s < sh.angles; ++s) {
      const int src = o.src[s], idx = o.idx[s];
      if (src == VQC_SRC_PARAM) {
        if (idx < 0 || idx >= P) {
          msg = at + "param index " + std::to_string(idx) + " out of range";
          return VQC_ERR_INVALID_ARG;
        }
      } else if (src == VQC_SRC_INPUT) {
        if (idx < 0 || idx >= F) {
          msg = at + "input index " + std::to_string(idx) + " out of range";
          return VQC_ERR_INVALID_ARG;
        }
      } else if (src != VQC_SRC_CONST) {
        msg = at + "unknown angle source " + std::to_string(src);
        return VQC_ERR_INVALID_ARG;
      }
      if (!std::isfinite(o.val[s])) {
        msg = at + (src == VQC_SRC_CONST ? "constant angle" : "angle offset") + " is not finite";
        return VQC_ERR_INVALID_ARG;
      }
      if (src != VQC_SRC_CONST && (!std::isfinite(o.mul[s]) || o.mul[s] == 0.f)) {
        msg = at + "angle scale (mul) must be finite and nonzero";
        return VQC_ERR_INVALID_ARG;
      }
    }
    lower_gate(o, plan);
  }
  fold_trailing_entanglers(plan);
  find_heads(plan);
  const int n_occ = (int)plan.occ_src.size();
  if (reg_bits != 0 && (reg_bits < 2 || reg_bits > 5)) {
    msg = "reg_bits must be 0 (default) or in [2, 5]";
    return VQC_ERR_INVALID_ARG;
  }
  const int nq = std::max(n, kDefaultRegBits);  // qubits >= n stay |0> and are never read
  plan.nq = nq;
  // 14-qubit tiles go through the streaming kernels: their adjoint holds 32
  // amplitudes per thread in 512 threads, which keeps psi and lambda in registers
  if (path == VQC_PATH_AUTO) path = nq < kMaxTileQubits ? VQC_PATH_RESIDENT : VQC_PATH_STREAM;
  if (path != VQC_PATH_RESIDENT && path != VQC_PATH_STREAM) {
    msg = "unknown path option";
    return VQC_ERR_INVALID_ARG;
  }
  if (path == VQC_PATH_RESIDENT && nq > kMaxTileQubits) {
    msg = "the resident path holds at most 14 qubits";
    return VQC_ERR_UNSUPPORTED;
  }
  if (path == VQC_PATH_STREAM && nq < kMaxTileQubits) {
    msg = "the streaming path needs at least 14 qubits (its tiles hold 14)";
    return VQC_ERR_UNSUPPORTED;
  }
  if (path == VQC_PATH_RESIDENT && reg_bits > 4) {
    msg = "reg_bits on the resident path must be 2, 3 or 4";
    return VQC_ERR_INVALID_ARG;
  }
  if (path == VQC_PATH_STREAM && reg_bits != 0 && reg_bits < 4) {
    msg = "reg_bits on the streaming path must be 4 or 5";
    return VQC_ERR_INVALID_ARG;
  }
  plan.path = path;
  const std::vector<Prim> rev(plan.prims.rbegin(), plan.prims.rend());
  int rc = 0;
  if (path == VQC_PATH_RESIDENT) {
    // default width: at least 64 threads per sample up to 8 qubits, 2^(n-3) from
    // 9 to 10, 16 amplitudes per thread from 11 on (measured on configurations
    // of 4, 8 and 12 qubits: small states are latency bound, so more threads win)
    plan.R = reg_bits ? reg_bits : nq <= 8 ? 2 : nq <= 10 ? 3 : kDefaultRegBits;
    plan.k = nq;
    plan.t = nq - plan.R;
    const int T = 1 << plan.t;
    plan.WG = std::max(64, T);
    plan.S = plan.WG / T;
    plan.G = T >= 64 ? plan.WG / 64 : plan.S;
    // initial mapping: registers get the first qubits the sweep needs there
    Mapping m;
    m.k = plan.k;
    m.nq = nq;
    for (int q = 0; q < kMaxQubits; ++q) m.q2p[q] = -1;
    {
      const std::vector<int> nn = next_need_table(plan.prims, nq);
      std::vector<int> qs(nq);
      for (int q = 0; q < nq; ++q) qs[q] = q;
      std::stable_sort(qs.begin(), qs.end(), [&](int x, int y) { return nn[x] < nn[y]; });
      std::vector<int> rest(qs.begin() + plan.R, qs.end());
      std::sort(rest.begin(), rest.end());
      for (int r = 0; r < plan.R; ++r) {
        m.p2q[r] = qs[r];
        m.q2p[qs[r]] = r;
      }
      for (size_t j = 0; j < rest.size(); ++j) {
        m.p2q[plan.R + j] = rest[j];
        m.q2p[rest[j]] = plan.R + (int)j;
      }
    }
    auto global_slot = [&](int occ) { return plan.occ_slot[occ]; };
    plan.start_off = append_map(m, plan.maps);
    // gates on lane bits 0..3 (one or two DPP moves per value): generated
    // kernels with 4 amplitudes per thread, where exchanges are not hidden.
    // Qubits on lane bits 4 and 5 still come to a register bit, by a permlane
    // swap (one instruction per two values).
    plan.lanes = (lane_gates && plan.R <= 2) ? std::min(plan.t, 4) : 0;
    const bool lazy = plan.R >= 2;
    rc = plan_sweep(lazy ? lazy_diagonals(plan.prims, plan) : plan.prims, nq, plan.k, plan.R, m,
                    plan.fwd, plan.cols, plan.fwd_exchanges, global_slot, msg, plan.lanes);
    if (rc < 0) return rc;
    plan.end_off = append_map(m, plan.maps);
    rc = plan_sweep(lazy ? lazy_diagonals(rev, plan) : rev, nq, plan.k, plan.R, m, plan.bwd,
                    plan.cols, plan.bwd_exchanges, global_slot, msg, plan.lanes);
    if (rc < 0) return rc;
    plan.bwd_end_off = append_map(m, plan.maps);
    // LDS: exchange buffer | angle table [occ][S] | gradient accumulators [slot][G]
    const size_t xbuf = (size_t)plan.WG * ((size_t)1 << plan.R) * 8;
    plan.lds_tab = xbuf;
    const size_t tab = align_up((size_t)n_occ * plan.S * 8, 16);
    plan.lds_acc = xbuf + tab;
    const size_t acc = align_up((size_t)(P + F) * plan.G * 4, 16);
    plan.lds_fwd = std::max<size_t>(xbuf + tab, 16);
    plan.lds_bwd = xbuf + tab + acc;
    // training step: E and g rows of the workgroup's samples after the adjoint's
    // tables
    plan.lds_e = align_up(plan.lds_bwd, 16);
    plan.lds_step = plan.lds_e + (2 * (size_t)plan.S * n + plan.S) * 4;  // E, g, targets
  } else {
    // Tiles of the generated kernels: 13 qubits unless tile_qubits says
    // otherwise (vqc_compile also plans 12 and keeps that plan when it takes at
    // most a quarter more passes).  Below 14 qubits several workgroups share a
    // CU and one's HBM traffic overlaps another's compute.  Measured: the
    // 16-qubit workload 63 k -> 77-81 k evals/s at 13 qubits despite more
    // passes; the 14-qubit one 512 k -> 534 k although its state no longer
    // fits one tile.
    plan.k = tile_qubits ? tile_qubits : lane_gates ? kMaxTileQubits - 1 : kMaxTileQubits;
    plan.ng = nq - plan.k;
    plan.Rf = reg_bits ? reg_bits : kStreamRegBitsFwd;
    plan.Rb = reg_bits ? reg_bits : kStreamRegBitsBwd;
    plan.t = plan.k - plan.Rf;       // the forward's geometry (informational)
    plan.WG = 1 << plan.t;
    plan.S = 1;
    plan.G = plan.WG / 64;
    rc = plan_stream_both(plan, msg);
    if (rc < 0) return rc;
    stream_lds(plan);
  }
  if (std::max(plan.lds_bwd, plan.lds_step) > (size_t)kLdsBytes) {
    msg = "circuit too large for on-chip tables: " +
          std::to_string(std::max(plan.lds_bwd, plan.lds_step)) +
          " bytes of LDS needed (limit " + std::to_string(kLdsBytes) + ")";
    return VQC_ERR_TOO_LARGE;
  }
  return 0;
}

// The streaming training step's plan: the passes of `full` planned again
// without the heads' rotations.  Its first forward pass starts from the
// product state after the heads, its last adjoint pass ends where the heads
// end and contracts lambda against the heads' states (the per-tile partials of
// the vectors v_q), and a last kernel sums those partials and takes the head
// rotations' gradients.  Returns 1 (and leaves `step` unspecified) when the
// circuit has no head rotation.
int build_step_plan(const Plan& full, Plan& step, std::string& msg) {
  if (full.path != VQC_PATH_STREAM) return 1;
  std::vector<char> in_head(full.occ_src.size(), 0);
  bool any = false;
  for (const auto& hq : full.head)
    for (const Prim& g : hq) {
      if (g.occ >= 65536) return 1;  // the head tables hold 16-bit occurrence numbers
      in_head[g.occ] = 1;
      any = true;
    }
  if (!any || full.n > 64) return 1;  // one lane per qubit walks its head
  if (full.P + full.F > kMaxStepSlots) return 1;  // the head kernel's LDS row of slots
  step = full;
  step.prims.clear();
  for (const Prim& g : full.prims)
    if (!(g.occ >= 0 && in_head[g.occ])) step.prims.push_back(g);
  step.fwd.clear();
  step.bwd.clear();
  step.cols.clear();
  step.maps.clear();
  step.pslots.clear();
  step.fpass.clear();
  step.bpass.clear();
  step.fwd_exchanges = step.bwd_exchanges = 0;
  step.max_pass_slots = 0;
  step.product_head = true;
  const int rc = plan_stream_both(step, msg);
  if (rc < 0) return rc;
  stream_lds(step);
  if (step.lds_bwd > (size_t)kLdsBytes) {
    msg = "circuit too large for on-chip tables";
    return VQC_ERR_TOO_LARGE;
  }
  return 0;
}

}  // namespace vqc
