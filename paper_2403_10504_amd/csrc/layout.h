// Host-side layout rules shared by the planner and the runtime: the tensor
// layout of each node's host range and the static carving of the device
// arena.  Pure C++; no HIP dependency.
#pragma once

#include <stdint.h>

#include <algorithm>
#include <string>
#include <vector>

#include "../../include/atom.h"

namespace atom {

constexpr uint64_t ALIGN = 256;
inline uint64_t align_up(uint64_t x, uint64_t a = ALIGN) { return (x + a - 1) / a * a; }
inline int64_t vocab_padded(int64_t V) { return (V + 127) / 128 * 128; }
inline int elem_bytes(const atom_config& c) { return c.dtype == ATOM_BF16 ? 2 : 4; }
// Rows of the logits chunk of the LM head (the [N][V] fp32 logits are never
// held whole).
constexpr int64_t HEAD_CHUNK = 2048;
// fp32 workspace that lets weight-gradient GEMMs of narrow layers split their
// long token dimension over workgroups.
constexpr uint64_t SPLITK_BYTES = 64ull << 20;
// Steps one pipelined call may run (one loss slot each).
constexpr int MAX_STEPS_PER_CALL = 64;
// Host checkpoints: block inputs live in a device ring of this many entries
// per micro-batch; the forward copies to the host every input the ring will
// overwrite (indices 0..L-CKPT_RING) and the backward restores them.
constexpr int CKPT_RING = 4;
inline int ckpt_evicted(const atom_config& c) { return c.ckpt == ATOM_CKPT_HOST ? std::max(0, c.n_layer + 1 - CKPT_RING) : 0; }
// Bytes of block inputs one step copies each way under host checkpoints.
inline uint64_t ckpt_xfer_bytes(const atom_config& c) {
  return static_cast<uint64_t>(ckpt_evicted(c)) * c.accum * static_cast<uint64_t>(c.batch) * c.seq_len * c.d_model * 4;
}

struct TensorDesc {
  std::string name;
  int64_t rows, cols;
  uint64_t offset, bytes;
};

// Tensors of node `node` with 256-byte aligned offsets; returns node bytes.
uint64_t node_tensors(const atom_config& c, int node, std::vector<TensorDesc>* out);

// Validation of a configuration; returns an empty string when usable.
std::string check_config(const atom_config& c);

// Offsets (bytes from the arena base) of every region of the device arena.
struct ArenaLayout {
  // reserve regions
  uint64_t tok_in, tok_tgt, emb_perm, emb_seg, emb_uniq;  // slot 0; slot 1 at + tok_stride
  uint64_t tok_stride;
  uint64_t ckpt, ckpt_bytes_each;  // (L+1) (host checkpoints: CKPT_RING) x accum x [N][d] fp32 block inputs
  uint64_t dres, dres_lp;          // accum x [N][d] fp32 / working dtype
  uint64_t loss_rows, loss_out;
  uint64_t hwm;                    // 8-byte counters of the working-memory probe (atom_profile_nodes)
  uint64_t splitk, splitk_bytes;   // fp32 workspace for GEMMs split over k
  uint64_t ws;                     // start of the union workspace
  // block workspace (offsets inside ws)
  uint64_t a, qkv, o, x1, c, u, g, mu1, rs1, mu2, rs2, lse, delta, du, dbuf, dout, dqkv, part;
  // head workspace (offsets inside ws)
  uint64_t yhat, fmu, frs, logits, dz, dyhat, hpart;
  uint64_t ws_bytes, part_floats;
  uint64_t block_ws, head_ws;      // workspace a block / the head uses (ws_bytes is the larger)
  uint64_t reserve_bytes;
  // slots (valid once a plan is known)
  uint64_t wslots, gslots, accslot;
  uint64_t arena_bytes;
};

ArenaLayout arena_layout(const atom_config& c, uint64_t slot_bytes, int n_slots, int n_gslots);

}  // namespace atom
