// Host-side model object and workspace of the DPA4C library.
#pragma once

#include <mutex>
#include <vector>

#include "common.h"

struct dpa4c_model;

namespace dpa4c {

enum Stage {
  kStNeighbor = 0,   // skin-list builds (count, fill, reverse index, snapshot)
  kStSkinRev,        // reverse index of a caller-built skin list
  kStForward,
  kStAtoms,
  kStBackward,
  kStForces,
  kStEnergy,
  kStIntegrate,
  kNumStages
};
const char* stage_name(int s);

// grow-only device buffer
// cell-list grid of a periodic cell (neighbors.hip, make_grid)
struct CellGrid {
  int64_t qh[9];      // lattice vectors in fixed point, row b = Q(h_b)
  double h[9];        // lattice vectors (A), row b = h_b
  double inv[9];      // inverse of the lattice matrix: fractional f = x inv
  int tric;           // 0: diagonal (orthorhombic) cell, binned in integers
  int nc[3];          // cells per axis
  int reach[3];       // stencil half width per axis
  int64_t rq;         // fixed-point neighbour radius
  int64_t ncell;
};

struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
  int ensure(size_t want);   // returns 0 or DPA4C_ERR_HIP
  void release();
  template <class T> T* as() const { return static_cast<T*>(p); }
};

// Cell-list scratch used by neighbour builds.
struct NeighborScratch {
  DevBuf qpos;       // int64 [N][3] wrapped fixed-point positions
  DevBuf wrap;       // int32 [N][3] lattice translations removed by wrapping
  DevBuf cell_of;    // int32 [N]
  DevBuf cell_cnt;   // int32 [ncell]
  DevBuf cell_start; // int32 [ncell+1]
  DevBuf cell_fill;  // int32 [ncell]
  DevBuf cell_rec;   // 32-byte records [N] in bin order: fixed-point position and atom index
  DevBuf long_keys;  // int64 [cap] keys of rows longer than the fill kernel's LDS row
  DevBuf counts;     // int64 [N]
  DevBuf partials;   // int64 scan partials
  DevBuf host_flag;  // pinned host int64 [4]
  DevBuf extent;     // int64 [6]: min and max of the fixed-point positions
  int64_t* host_extent = nullptr;   // pinned [6]
};

struct Workspace {
  int64_t n_atoms = 0;
  int64_t cap = 0;
  // skin list owned by verlet_step
  DevBuf skin_row;      // int64 [N+1]
  DevBuf skin_j;        // int32 [cap]
  DevBuf skin_shift;    // int32 [cap]
  DevBuf skin_rev;      // int64 [cap]: position in the list of the reverse edge, or -1
  DevBuf qbuild;        // int64 [N][3] fixed-point positions at the last build
  // compacted (r < r_c) edges, stored in the rows of the skin list
  DevBuf ecount;        // int32 [N]
  DevBuf edge;          // float4 [cap]: r_ij (x, y, z) and j (bits)
  DevBuf cskin;         // int32 [cap]: skin position of each compact slot (row-local)
  DevBuf watom;         // double [N][9]: per-centre virial terms (when not the caller's)
  // per-atom state
  DevBuf node;          // float [N][NS]
  DevBuf node_grad;     // float [N][NS]: dE/d(node state)
  DevBuf desc;          // float [N][D_out]: D, written only for stage checks
  DevBuf epart;         // double partial sums
  DevBuf flags;         // int64 [8] device flags
  DevBuf eatom;         // double [N] (per-atom energies inside verlet_step)
  DevBuf tailpart;      // double [2][2][groups]: energy partials of a Verlet step
  DevBuf virpart;       // double [2][groups][9]: virial partials
  DevBuf nvt;           // double: chain state of an NVT call and its batch backup
  DevBuf backup;        // double [3][N][3]: positions, velocities, forces at a batch start
  DevBuf inv_mass;      // double [T+1]: 1 / (m * 103.6427)  (A/fs^2 per eV/A)
  DevBuf mass;          // double [T+1]
  int64_t* host_flags = nullptr;          // pinned [8]
  // pair-folded tables of the species present (fold.hip)
  DevBuf ftab;          // float [fold_n^2][n_rows][C0 * kFoldWords]
  DevBuf fold_map;      // int32 [T+1]: type -> folded index, or -1
  DevBuf fold_mask;     // uint32 [4]: species present in the last call
  DevBuf fidx;          // int32 [N]: folded index of every atom
  DevBuf check;         // int64 [2]: reverse pairs found in a caller's list
  // pinned host words, allocated with the model: [0, 16) the species
  // presence mask, [16, 32) row_ptr[N] and the reverse pairs of a caller's
  // list, [64, 64 + 4 (T+1)) the type map of the folded tables
  uint32_t* fold_host = nullptr;
  // inputs of the last evaluation (the stage-check entry point re-runs it)
  const int32_t* last_species = nullptr;
  const int32_t* last_fidx = nullptr;     // folded index of that call, or null (separable)
  const double* last_pos = nullptr;
  const int64_t* skin_row_used = nullptr;
  const int32_t* skin_j_used = nullptr;
  const int32_t* skin_shift_used = nullptr;
  int64_t cap_used = 0;
  CellGrid last_grid{};
  // the dynamics' skin list as left by the last call (periodic cells only):
  // valid for a call with the same atom count, cell and list radius (the
  // displacement check against qbuild decides whether it still covers the
  // positions); any other use of the reverse-index buffers clears it
  bool list_valid = false;
  int64_t list_n = 0, list_rq = 0, list_steps_since_build = 0;
  double list_cell[9] = {};
  NeighborScratch nb;
};

struct Timing {
  int64_t mask = 0;               // stages (bit s = stage s) that record events
  std::vector<hipEvent_t> pool;
  std::vector<int> ev_stage;      // stage of each recorded pair
  size_t used = 0;
  double ms[kNumStages] = {};
  int64_t count[kNumStages] = {};
};

}  // namespace dpa4c

struct dpa4c_model {
  int device = 0;
  int C0 = 0, L = 0, R = 0, n_rbf = 0, F = 0, n_layers = 0, n_types = 0;
  double r_c = 0, delta = 0;
  int C[5] = {}, K[5] = {};
  int S = 0, D_out = 0, H = 0, Hp = 0, n_rows = 0;
  // device parameter storage
  dpa4c::DevBuf params;             // one allocation holding every array below
  float* gtab = nullptr;
  float* qtab = nullptr;
  float* pair = nullptr;
  float* type_embed = nullptr;
  float* W1 = nullptr;
  float* W2 = nullptr;
  float* A1 = nullptr;
  float* A2 = nullptr;
  float* mu = nullptr;
  float* inv_sigma = nullptr;
  float* E_ref = nullptr;
  float* theta[8] = {};             // Theta_t [in][F]
  float* thetaT[8] = {};            // Theta_t^T [F][in]
  float* bias[8] = {};
  float* wfrag[8] = {};             // Theta_t in MFMA fragment order
  float* wfragT[8] = {};            // Theta_t^T in MFMA fragment order
  float* w_head = nullptr;
  float b_head = 0;
  float* cpl = nullptr;             // dense (1,2,3) and (2,3,3) couplings (degree three only)
  // host copies kept for tests of the host logic
  std::vector<double> gaunt[4];     // (1,1,2), (1,2,3), (2,2,2), (2,3,3) normalised couplings
  dpa4c::Workspace ws;
  dpa4c::Timing timing;
  std::mutex mu_lock;
  int64_t last_n = 0;
  int fold_n = -1;                  // species with folded tables; 0 = separable path, -1 = unset
  float c_scale[4] = {1.0f, 1.0f, 1.0f, 1.0f};   // float16 scales of c2 .. c5 (folded tables use c2, c3)
  // the folded tables hold c0, c1, c2, c3: the float16 rounding of c2, c3
  // and the dropped c4, c5 are within bounds (else separable tables only)
  bool fold_allowed = true;
  uint32_t fold_types_mask[4] = {};

  dpa4c::ModelDev dev() const;
};
