// Internal interface between the C-ABI host code and the gfx950 kernels.
#ifndef FABFT_KERNELS_H
#define FABFT_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fabft {

// Query rows per workgroup for head dimension d: 8 waves of 32 rows, or 4
// waves at d = 256 (one wave per SIMD, for the register file of 512).
constexpr int query_tile_for(int d) { return d == 256 ? 128 : 256; }

// One injected single-bit fault (site numbers and fields as fabft_fault,
// with the head flattened to bh = b * H + h).
constexpr int kMaxFaults = 8;
struct FaultDesc {
  int site, bh, row, col, tile, bit;
};

struct FwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* resid;
  uint8_t* flags;
  float* pred;    // injection/debug kernels only; may be null
  float* actual;  // injection/debug kernels only; may be null
  float* pred_w;    // weighted check, debug kernels only; may be null
  float* actual_w;  // weighted check, debug kernels only; may be null
  // score check, debug kernels only; may be null: the row's sum of raw
  // scores over the key tiles without a mask (lhs), q_i . sum_k K_k over the
  // same keys (rhs) and |q_i| . sum_k |K_k| (the bound); 0 with the check off
  float* s_lhs;
  float* s_rhs;
  float* s_bound;
  int wcheck;     // 1: also run the weighted (alternating-sign) checksum
  // split over the keys (mode 3): workgroup (head, query tile, split) runs
  // key tiles [split*split_tiles, (split+1)*split_tiles) and writes the
  // partial state of each row to ws (see launch_merge)
  int nsplit;
  int split_tiles;
  float* ws;
  int dio;               // head dimension of q, k, v, o in memory (<= the
                         // kernel's width; the rest of the width is zero)
  // score check (modes 1, 2; null = off): per head, ntk + 1 rows of the
  // kernel's width D, the exclusive prefix over key tiles of the column sums
  // of K (kpre) and of |K| (kabs); tau_s its relative threshold
  const float* kpre;
  const float* kabs;
  int ntk;
  float tau_s;
  int Lq, Lk;
  int n_qt;       // query tiles per head
  int n_items;    // work items (head, query tile): B * H * n_qt
  int grid;       // workgroups: n_items (times nsplit in mode 3), or fewer
                  // with persist
  int persist;    // 1: each of the grid's workgroups runs a list of items
                  // (set by launch_fwd, modes 0 and 1 only)
  float sl2;      // scale * log2(e)
  float tau_rel, tau_abs;
  int nf;                          // faults in f (injection kernels only)
  FaultDesc f[kMaxFaults];
};

// mode 0: checksum off, 1: checksum on, 2: checksum on + debug/injection,
// 3: checksum on, one key split per workgroup (partial states to p.ws),
// 4: checksum on, two passes over the keys (Algorithm 1: the row max first),
// 5: mode 4 with injection/debug outputs.
// Modes 0 and 1 (without the score check) may run as many workgroups as fit
// on the device at once, each running a list of items, when there are more
// items than that (set_persistent: off, automatic, always).
int launch_fwd(const FwdParams& p, int d, bool causal, int mode, hipStream_t stream);
enum { kPersistOff = 0, kPersistAuto = 1, kPersistAlways = 2 };
void set_persistent(int mode);
int get_persistent();
int key_tile(int d);
// Width the kernels compute with for a head dimension d (64, 96, 128 or
// 256): d itself, or 128 for d = 96 (columns 96..127 are zero on chip).
inline int compute_width(int d) { return d == 96 ? 128 : d; }
// Partial-state record of (head, row, split) in the split workspace, in
// floats: m (exp2 domain), l, c, c_w, then the d unnormalised outputs o.
inline int split_record_floats(int d) { return d + 4; }
// Merge the partial states of every row (mode 3 writes them) into O, resid
// and flags.
int launch_merge(const FwdParams& p, int d, int nheads, hipStream_t stream);
// Column sums of K per key tile and their exclusive prefix over the tiles
// (kpre) and the same for |K| (kabs): BH heads, (ceil(Lk/64) + 1) rows of
// compute_width(d) floats each.
int launch_kpre(const uint16_t* k, int BH, int Lk, int d, float* kpre, float* kabs,
                hipStream_t stream);
inline long long kpre_floats(long long BH, int Lk, int d) {
  return BH * ((Lk + 63) / 64 + 1) * (long long)compute_width(d);
}
int launch_head_flags(const uint8_t* flags, int BH, int Lq, uint8_t* hflags, hipStream_t stream);
int launch_global(const uint16_t* o, const float* resid, int BH, int Lq, int d, float tau_rel,
                  float tau_abs, double* gsum, uint8_t* gflag, hipStream_t stream);

}  // namespace fabft

#endif
