// Kernel launchers (defined in the .hip sources) called by the host code.
#pragma once

#include "compact.h"
#include "model.h"

namespace dpa4c {

// host-only checks of a weight blob's header (no device is touched)
int check_blob_header(const void* blob, size_t nbytes);
int create_model(const void* blob, size_t nbytes, int device, dpa4c_model** out);
int launch_pair_cache(dpa4c_model* m, const float* wp_in, const float* wp_out);

// neighbour lists (orthorhombic, periodic); all on ``st``
// (CellGrid: model.h)
int make_grid(const double cell[9], int64_t rq, CellGrid* g);
// bin, count and scan (row_ptr); flags[3] receives the longest row (an
// atomic maximum: the caller clears it)
int build_skin_list(NeighborScratch& nb, const double* pos, int64_t n, const CellGrid& g,
                    int64_t* row_ptr, int64_t* flags, hipStream_t st);
// the sorted rows of a counted list; ``max_row`` (the longest row, from the
// count) above the LDS row size makes the fill use a global scratch for
// those rows.  With ``jsamp`` (int32 [cap / 16 + 1]) the neighbour index at
// every 16th position of the list also goes there for launch_skin_rev.
int fill_skin_list(NeighborScratch& nb, int64_t n, const CellGrid& g, const int64_t* row_ptr,
                   int32_t* nbr_j, int32_t* nbr_shift, int64_t cap, int64_t* flags,
                   int64_t max_row, int32_t* jsamp, hipStream_t st);
// per-axis min and max of the fixed-point positions Q(x) (finite ones):
// host6 = [min x, y, z, max x, y, z]; dev6 is device scratch of 6 int64;
// synchronises ``st``
int position_extent(const double* pos, int64_t n, int64_t* dev6, int64_t* host6, hipStream_t st);
// skin_rev[s] = position in the list of the reverse of skin edge s (in row
// nbr_j[s]), or -1;
// jsamp = scratch of cap / 16 + 1 int32: nbr_j at every 16th position of the
// list, computed here unless ``jsamp_ready`` (fill_skin_list wrote it);
// with ``paired`` (device int64, zeroed by the caller) also the number of
// reverse pairs found, so a symmetric list of E entries gives E / 2; with
// ``order_of`` (the scratch of the build that made this list) the rows are
// taken in the build's spatial bin order
struct NeighborScratch;
int launch_skin_rev(const int64_t* row_ptr, const int32_t* nbr_j, const int32_t* nbr_shift,
                    int64_t n, int64_t cap, int32_t* jsamp, bool jsamp_ready, int64_t* skin_rev,
                    int64_t* paired, const NeighborScratch* order_of, hipStream_t st);
// species analysis of a call: builds the pair-folded tables of the species
// present when they changed (at most kMaxFoldTypes species) and the folded
// index of every atom into ``fidx`` [n]; ``mask_dev`` is device scratch of 4
// uint32.  Without ``may_alloc`` the tables are rebuilt only inside the
// allocation they already have; a species set that needs more runs this call
// on the separable tables and leaves the model's folded state as it was.
// *use_fold tells the edge kernels which tables to read.  Synchronises ``st``.
int prepare_species(dpa4c_model* m, const int32_t* species, int64_t n, uint32_t* mask_dev,
                    int32_t* fidx, bool may_alloc, bool* use_fold, hipStream_t st);

// model stages: the edge kernels read the pair-folded tables with the
// folded index ``fidx`` of every atom, or the separable tables when fidx is null
// compaction of every skin row (compact.h) and the forward pass
int launch_forward(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
                   const int64_t* row_ptr, const CompactArgs& ca, float* node, hipStream_t st);
// readout + MLP + head + MLP gradient + readout VJP on 16-atom tiles;
// desc_out (float [N][D_out]) receives D when not null
int launch_atoms(const dpa4c_model* m, int64_t n, const int32_t* species, const float* node,
                 float* node_grad, double* e_atom, float* desc_out, hipStream_t st);
// the gradient dE/dr_ij of compact slot c of row i goes to the skin position
// of that edge, edge[row_ptr[i] + cskin[row_ptr[i] + c]] (x, y, z = the
// gradient, w = the bits of j as before), over the compact records, which
// it reads first; with w_atom ([N][9]) also the virial terms
// W_i = -sum_e g_e (x) r_e of every centre
int launch_backward(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
                    const int64_t* row_ptr, const int32_t* ecount, float4* edge,
                    const int32_t* cskin, const float* node_grad, double* w_atom, hipStream_t st);
struct StepTail;
// the virial of Eq. (forces): atom = [N][9] per-centre terms W_i written by
// the backward kernel, part_v = [tail_partial_count(n)][9] block partials of
// them summed in a fixed order by the force assembly
struct VirialOut {
  double* part_v;
  double* atom;
};
// force assembly; with ``tail`` also the velocity-Verlet work of the step
// that needs only F_k (see StepTail), with ``vir`` the virial
int launch_forces(int64_t n, const int64_t* row_ptr, const int32_t* ecount, const float4* grad,
                  const int32_t* cskin, const int64_t* skin_rev,
                  double* forces, const StepTail* tail, const VirialOut* vir, hipStream_t st);
// out[c] = fixed-order sum over p < np of part[ncomp p + c]
int launch_sum_components(const double* part, int64_t np, int ncomp, double* out, hipStream_t st);
int launch_energy(int64_t n, const double* e_atom, double* partials, double* out,
                  hipStream_t st);

// dense fp32 GEMM on MFMA for tests of the kernel itself
int launch_gemm_test(const float* A, const float* B, float* C, int M, int N, int K,
                     hipStream_t st);

// velocity Verlet pieces
// block partials of a step's energies and where their totals go (np = 0:
// nothing to add)
struct StepSums {
  const double* part_e;
  const double* part_k;
  int np;
  double* e_pot;
  double* e_kin;
};
// The velocity-Verlet work fused into the force assembly of a step: the
// second half kick, the block partials of E_pot and E_kin (tail_partial_count(n)
// of each) and, with kick_next, the first half kick and the drift of step
// next_step with its displacement check against qbuild (none when null).
// An extra block writes the totals of ``prev``, whose partials must be a
// different buffer from part_e/part_k.
struct StepTail {
  double* pos;
  double* vel;
  const int32_t* species;
  const double* inv_mass;
  const double* mass;
  int n_types1;
  double half_dt, dt;
  const double* e_atom;
  double* part_e;
  double* part_k;
  StepSums prev;
  int kick_next;
  const int64_t* qbuild;
  int64_t skin_q;
  int64_t* flags;
  int64_t next_step;
};
// half kick (and drift with the displacement check of step ``step`` when
// qbuild is given), after v *= *scale when scale is not null; block 0 first
// adds the partials of the previous step
int launch_kick_drift(double* pos, double* vel, const double* forces, const int32_t* species,
                      const double* inv_mass, int n_types1, int64_t n, double dt, int drift,
                      const int64_t* qbuild, int64_t skin_q, int64_t* flags, StepSums prev,
                      int64_t step, const double* scale, hipStream_t st);

// Nose-Hoover chain (NVT): one launch closes a step (its chain half step,
// kinetic, potential and thermostat energies and virial, from the step's
// partials) and/or opens the next (the chain half step at the current
// kinetic energy); state = [xi_1..M, v_1..M, velocity scale to apply]
constexpr int kMaxChain = 8;
struct NhcArgs {
  double* state;
  int M;
  double kT, nf, dt;        // kT (eV), N_f, time step (fs)
  double Q[kMaxChain];      // chain masses (eV fs^2)
  const double* part_k;     // kinetic-energy partials [np]
  const double* part_e;     // potential-energy partials [np] (closing only)
  const double* part_v;     // virial partials [np][9] (closing only)
  int64_t np;
  int close_prev, open_next;
  double* e_pot;            // outputs of the closed step, each may be null
  double* e_kin;
  double* e_thermo;
  double* virial;           // [9]
};
int launch_nhc(const NhcArgs& a, hipStream_t st);
// kinetic-energy partials of the current velocities (kinetic_partial_count(n))
int kinetic_partial_count(int64_t n);
int launch_kinetic(const double* vel, const int32_t* species, const double* mass, int n_types1,
                   int64_t n, double* part_k, hipStream_t st);
// vel *= *scale
int launch_scale(double* vel, int64_t n, const double* scale, hipStream_t st);
int launch_final_step(StepSums prev, hipStream_t st);
// blocks of the force assembly, each writing one partial of the step's
// E_pot and E_kin (and virial): min(ceil(n/16), kMaxTailBlocks)
constexpr int kMaxTailBlocks = 8192;
int tail_partial_count(int64_t n);
int launch_snapshot_q(const double* pos, int64_t n, int64_t* qbuild, hipStream_t st);
// p[0, n) = 0 (a fill kernel, not a memset node)
int launch_zero_i64(int64_t* p, int64_t n, hipStream_t st);

// The per-call device buffers of an energy-and-force evaluation: the
// model's workspace, or a caller-free scratch area (noalloc.hip).
struct EvalBufs {
  int32_t* ecount;      // int32 [N]
  float4* edge;         // float4 [cap]
  int32_t* cskin;       // int32 [cap]
  int64_t* skin_rev;    // int64 [cap]
  float* node;          // float [N][S+2]
  float* node_grad;     // float [N][S+2]
  double* epart;        // double [partial_count(N) + 8]
  int32_t* fidx;        // int32 [N]
  uint32_t* fold_mask;  // uint32 [4]
  int64_t* check;       // int64 [2]: reverse pairs found
};
// bytes of each EvalBufs array for N atoms, a list of cap entries and a node
// state of ns floats per atom, each rounded up to 256 (in struct order)
constexpr int kEvalBufs = 10;
void eval_buf_sizes(int64_t n, int64_t cap, int ns, size_t sizes[kEvalBufs]);
// compute_energy_forces(_virial) on the given buffers (null: the model's
// workspace, grown as needed); ``bufs`` given means no allocation, no timing
// events and no memset nodes on the stream
int energy_forces_core(const dpa4c_model* m, const double* pos, const int32_t* species, int64_t N,
                       const double cell[9], const int pbc[3], double r_c, const int64_t* row_ptr,
                       const int32_t* nbr_j, const int32_t* nbr_shift, int64_t n_pairs,
                       double* e_atom, double* forces, double* e_total, double* virial,
                       double* atom_virial, const EvalBufs* bufs, void* stream);
// per-device set-up of the no-allocation entry point (noalloc.hip); called
// with ``device`` current by dpa4c_model_create
int noalloc_setup(int device);
// flags[idx] = value
int launch_set_flag(int64_t* flags, int idx, int64_t value, hipStream_t st);
int partial_count(int64_t n);

}  // namespace dpa4c
