// C-ABI entry points of the DPA4C library (declared in include/dpa4c.h).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>

#include "../../include/dpa4c.h"
#include "launch.h"
#include "model.h"

namespace dpa4c {

namespace {
thread_local std::string g_last_error;

// per-device scratch of build_neighbors
std::mutex g_nb_lock;
std::map<int, NeighborScratch*> g_nb_scratch;
std::map<int, DevBuf*> g_nb_flags;

constexpr int64_t kFlagCapacity = 1, kFlagRowTooLong = 2, kFlagShift = 4, kFlagNonFinite = 8;

// Periodicity of a call.  A null cell is an open system (every axis open);
// with a cell, pbc[a] = 0 opens axis a, which needs an orthorhombic
// (diagonal) cell.
struct CellSpec {
  double cell[9];
  bool open[3];
  bool any_open;
};

int cell_spec(const double* cell, const int* pbc, CellSpec* cs) {
  cs->any_open = false;
  for (int k = 0; k < 9; ++k) cs->cell[k] = (k % 4 == 0) ? 1.0 : 0.0;
  if (!cell) {
    for (int a = 0; a < 3; ++a) cs->open[a] = true;
    cs->any_open = true;
    return 0;
  }
  if (!pbc) {
    set_error("pbc must not be null when a cell is given");
    return DPA4C_ERR_INVALID_ARG;
  }
  for (int a = 0; a < 3; ++a) {
    cs->open[a] = pbc[a] == 0;
    cs->any_open = cs->any_open || cs->open[a];
  }
  for (int k = 0; k < 9; ++k) cs->cell[k] = cell[k];
  if (cs->any_open) {
    for (int a = 0; a < 3; ++a)
      for (int b = 0; b < 3; ++b)
        if (a != b && cell[3 * a + b] != 0.0) {
          set_error("open (non-periodic) axes need an orthorhombic cell");
          return DPA4C_ERR_UNSUPPORTED;
        }
    for (int a = 0; a < 3; ++a)
      if (cs->open[a]) cs->cell[4 * a] = 1.0;   // replaced by effective_cell
  }
  return 0;
}

// The lattice a build or an evaluation uses.  An open axis gets the virtual
// length extent + 2 r + 1 A: no image of any atom then lies within r along
// it, so the periodic machinery yields exactly the open-boundary neighbours
// (image index 0 on that axis).  The extent (max - min of the positions
// along the axis) is read from the device when ``pos`` is given; without it
// the length is a placeholder, which compaction never uses (it multiplies
// the lattice vector of an open axis by its image index, 0).
int effective_cell(const CellSpec& cs, const double* pos, int64_t n, double r, NeighborScratch& nb,
                   hipStream_t st, double out[9]) {
  for (int k = 0; k < 9; ++k) out[k] = cs.cell[k];
  if (!cs.any_open) return 0;
  double ext[3] = {0.0, 0.0, 0.0};
  if (pos && n > 0) {
    DPA4C_TRY(nb.extent.ensure(6 * sizeof(int64_t)));
    if (!nb.host_extent)
      DPA4C_HIP_TRY(hipHostMalloc((void**)&nb.host_extent, 6 * sizeof(int64_t), hipHostMallocDefault));
    int rc = position_extent(pos, n, nb.extent.as<int64_t>(), nb.host_extent, st);
    if (rc) return rc;
    for (int a = 0; a < 3; ++a)
      if (nb.host_extent[3 + a] >= nb.host_extent[a])
        ext[a] = double(nb.host_extent[3 + a] - nb.host_extent[a]) / kQScale;
  }
  for (int a = 0; a < 3; ++a)
    if (cs.open[a]) {
      out[4 * a] = ext[a] + 2.0 * r + 1.0;
      if (out[4 * a] > 1.0e6) {
        set_error("an open system wider than 1e6 A");
        return DPA4C_ERR_UNSUPPORTED;
      }
    }
  return 0;
}

int64_t qfix_host(double x) { return static_cast<int64_t>(std::rint(x * kQScale)); }

int flags_to_error(int64_t f) {
  if (f & kFlagNonFinite) {
    set_error("non-finite (or |x| > 1e12) position");
    return DPA4C_ERR_NONFINITE;
  }
  if (f & kFlagRowTooLong) {
    set_error("a neighbour row is longer than the fill kernel's row buffer and no scratch was given");
    return DPA4C_ERR_UNSUPPORTED;
  }
  if (f & kFlagShift) {
    set_error("an image index exceeds +-127 (atom far outside the cell)");
    return DPA4C_ERR_UNSUPPORTED;
  }
  if (f & kFlagCapacity) {
    set_error("neighbour capacity exceeded");
    return DPA4C_ERR_CAPACITY;
  }
  return 0;
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    hipGetDevice(&prev);
    if (prev != dev) hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur;
    hipGetDevice(&cur);
    if (prev >= 0 && cur != prev) hipSetDevice(prev);
  }
};

// Stage timing with HIP events on the caller's stream.
struct StageScope {
  dpa4c_model* m;
  hipStream_t st;
  int stage;
  size_t slot = SIZE_MAX;
  StageScope(const dpa4c_model* mm, int s, hipStream_t stream, bool on = true)
      : m(const_cast<dpa4c_model*>(mm)), st(stream), stage(s) {
    if (!on || !m || !((m->timing.mask >> s) & 1)) return;
    Timing& t = m->timing;
    if (t.used + 2 > t.pool.size()) {
      size_t grow = t.pool.size() < 256 ? 256 : t.pool.size();
      for (size_t k = 0; k < grow; ++k) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        t.pool.push_back(e);
      }
      t.ev_stage.resize(t.pool.size() / 2);
    }
    slot = t.used;
    t.used += 2;
    t.ev_stage[slot / 2] = stage;
    hipEventRecord(t.pool[slot], st);
  }
  ~StageScope() {
    if (slot != SIZE_MAX) hipEventRecord(m->timing.pool[slot + 1], st);
  }
};

void collect_timing(dpa4c_model* m) {
  Timing& t = m->timing;
  if (!t.used) return;
  hipDeviceSynchronize();
  for (size_t s = 0; s + 1 < t.used; s += 2) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.pool[s], t.pool[s + 1]) == hipSuccess) {
      t.ms[t.ev_stage[s / 2]] += ms;
      t.count[t.ev_stage[s / 2]] += 1;
    }
  }
  t.used = 0;
}

// Workspace sizing for N atoms and a skin list of ``cap`` edges.
int ensure_workspace(dpa4c_model* m, int64_t n, int64_t cap) {
  Workspace& w = m->ws;
  const int64_t nn = n < 1 ? 1 : n, cc = cap < 1 ? 1 : cap;
  DPA4C_TRY(w.ecount.ensure(4 * nn));
  DPA4C_TRY(w.edge.ensure(16 * cc));
  DPA4C_TRY(w.cskin.ensure(4 * cc));
  DPA4C_TRY(w.skin_rev.ensure(8 * cc));
  DPA4C_TRY(w.node.ensure(4 * nn * (m->S + 2)));
  DPA4C_TRY(w.node_grad.ensure(4 * nn * (m->S + 2)));
  DPA4C_TRY(w.epart.ensure(8 * (partial_count(nn) + 8)));
  DPA4C_TRY(w.flags.ensure(8 * 8));
  DPA4C_TRY(w.eatom.ensure(8 * nn));
  DPA4C_TRY(w.fidx.ensure(4 * nn));
  DPA4C_TRY(w.fold_mask.ensure(4 * sizeof(uint32_t)));
  DPA4C_TRY(w.check.ensure(2 * sizeof(int64_t)));
  return 0;
}

// the model workspace as the buffers of an evaluation
EvalBufs ws_bufs(Workspace& w) {
  EvalBufs b{};
  b.ecount = w.ecount.as<int32_t>();
  b.edge = w.edge.as<float4>();
  b.cskin = w.cskin.as<int32_t>();
  b.skin_rev = w.skin_rev.as<int64_t>();
  b.node = w.node.as<float>();
  b.node_grad = w.node_grad.as<float>();
  b.epart = w.epart.as<double>();
  b.fidx = w.fidx.as<int32_t>();
  b.fold_mask = w.fold_mask.as<uint32_t>();
  b.check = w.check.as<int64_t>();
  return b;
}

// the compaction inputs and outputs of a model evaluation
CompactArgs compact_args(const CellGrid& g, const double* pos, const int32_t* nbr_j,
                         const int32_t* nbr_shift, int64_t rcq, int64_t cap, const EvalBufs& w) {
  CompactArgs ca{};
  ca.pos = pos;
  ca.nbr_j = nbr_j;
  ca.nbr_shift = nbr_shift;
  for (int k = 0; k < 9; ++k) {
    ca.qh[k] = g.qh[k];
    ca.h[k] = g.h[k];
  }
  ca.rcq = rcq;
  ca.tric = g.tric;
  ca.cap = cap;
  ca.ecount = w.ecount;
  ca.edge = w.edge;
  ca.cskin = w.cskin;
  return ca;
}

// NVT parameters of a dynamics call (nvt_step)
struct NvtConfig {
  double temperature;   // K
  double t_damp;        // fs
  int length;           // chain length M
  double* chain;        // device [2M]: xi_1..M then v_1..M, in/out
  double* e_thermo;     // device [nsteps]
  double* virial;       // device [nsteps][9] or null
};

// Everything after the skin list: forward (with the compaction of the skin
// rows), per-atom kernel, backward, forces and the energy sum, on the
// buffers ``B``; ``fidx`` is the folded index of every atom (null: the
// separable tables).  ``record``: the buffers are the model's workspace, so
// the stages may be timed and the inputs are kept for dpa4c_debug_stages.
int run_model(const dpa4c_model* mc, const double* pos, const int32_t* species, int64_t n,
              const CellGrid& g, const int64_t* row_ptr, const int32_t* nbr_j,
              const int32_t* nbr_shift, int64_t cap, const int64_t* skin_rev, double* e_atom,
              double* forces, double* e_total, const StepTail* tail, const VirialOut* vir,
              double* virial, const EvalBufs& B, const int32_t* fidx, bool record,
              hipStream_t st) {
  // e_total == nullptr: the caller sums the energy itself; ``tail``: the
  // velocity-Verlet work fused into the force assembly; ``vir``: the virial
  // partials (and per-atom terms), summed into virial[9] when that is given
  dpa4c_model* m = const_cast<dpa4c_model*>(mc);
  Workspace& w = m->ws;
  const int64_t rcq = qfix_host(m->r_c);
  int rc;
  const CompactArgs ca = compact_args(g, pos, nbr_j, nbr_shift, rcq, cap, B);
  {
    StageScope t(m, kStForward, st, record);
    rc = launch_forward(m, n, species, fidx, row_ptr, ca, B.node, st);
    if (rc) return rc;
  }
  {
    StageScope t(m, kStAtoms, st, record);
    rc = launch_atoms(m, n, species, B.node, B.node_grad, e_atom, nullptr, st);
    if (rc) return rc;
  }
  {
    StageScope t(m, kStBackward, st, record);
    rc = launch_backward(m, n, species, fidx, row_ptr, B.ecount, B.edge, B.cskin, B.node_grad,
                         vir ? vir->atom : nullptr, st);
    if (rc) return rc;
  }
  {
    StageScope t(m, kStForces, st, record);
    // the backward kernel has left dE/dr_ij in the edge array at the skin positions
    rc = launch_forces(n, row_ptr, B.ecount, B.edge, B.cskin, skin_rev, forces, tail, vir, st);
    if (rc) return rc;
    if (vir && virial) {
      rc = launch_sum_components(vir->part_v, tail_partial_count(n), 9, virial, st);
      if (rc) return rc;
    }
  }
  if (e_total) {
    StageScope t(m, kStEnergy, st, record);
    rc = launch_energy(n, e_atom, B.epart, e_total, st);
  }
  if (!record) return rc;
  m->last_n = n;
  w.last_species = species;
  w.last_fidx = fidx;
  w.last_pos = pos;
  w.last_grid = g;
  w.skin_row_used = row_ptr;
  w.skin_j_used = nbr_j;
  w.skin_shift_used = nbr_shift;
  w.cap_used = cap;
  return rc;
}

}  // namespace

void set_error(const std::string& msg) { g_last_error = msg; }

}  // namespace dpa4c

using namespace dpa4c;

extern "C" {

int dpa4c_model_create(const void* blob, size_t nbytes, int device, dpa4c_model** out) {
  if (!out) {
    set_error("dpa4c_model_create: null blob/out or blob shorter than its header");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (int rc = check_blob_header(blob, nbytes)) return rc;   // before any device call
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) {
    set_error("dpa4c_model_create: no such HIP device");
    return DPA4C_ERR_INVALID_ARG;
  }
  DeviceGuard guard(device);
  int rc = create_model(blob, nbytes, device, out);
  if (rc) return rc;
  // the species buffers every evaluation uses, allocated here so that the
  // entry point without allocation finds them
  Workspace& w = (*out)->ws;
  const size_t T1 = size_t((*out)->n_types) + 1;
  if (w.fold_map.ensure(4 * T1) != 0 ||
      hipHostMalloc((void**)&w.fold_host, 64 + 4 * T1, hipHostMallocDefault) != hipSuccess) {
    w.fold_host = nullptr;
    set_error("dpa4c_model_create: allocation of the species buffers failed");
    dpa4c_model_destroy(*out);
    *out = nullptr;
    return DPA4C_ERR_HIP;
  }
  rc = noalloc_setup(device);
  if (rc) {
    dpa4c_model_destroy(*out);
    *out = nullptr;
  }
  return rc;
}

void dpa4c_model_destroy(dpa4c_model* m) {
  if (!m) return;
  DeviceGuard guard(m->device);
  hipDeviceSynchronize();
  m->params.release();
  Workspace& w = m->ws;
  DevBuf* bufs[] = {&w.skin_row, &w.skin_j, &w.skin_shift, &w.skin_rev, &w.qbuild, &w.ecount,
                    &w.edge,     &w.cskin,  &w.node,
                    &w.desc,     &w.node_grad, &w.epart,  &w.flags,      &w.inv_mass, &w.mass,
                    &w.eatom,    &w.tailpart,  &w.backup,  &w.ftab,      &w.fold_map, &w.fold_mask,  &w.fidx,
                    &w.check,
                    &w.nb.qpos,  &w.nb.wrap, &w.nb.cell_of, &w.nb.cell_cnt, &w.nb.cell_start,
                    &w.nb.cell_fill, &w.nb.cell_rec, &w.nb.long_keys, &w.nb.counts,
                    &w.nb.partials,
                    &w.virpart,  &w.nvt,     &w.watom,     &w.nb.extent};
  for (DevBuf* b : bufs) b->release();
  for (hipEvent_t e : m->timing.pool) hipEventDestroy(e);
  if (w.host_flags) hipHostFree(w.host_flags);
  if (w.fold_host) hipHostFree(w.fold_host);
  if (w.nb.host_extent) hipHostFree(w.nb.host_extent);
  if (w.nb.host_flag.p) hipHostFree(w.nb.host_flag.p);
  delete m;
}

int dpa4c_model_info(const dpa4c_model* m, int64_t* info) {
  if (!m || !info) {
    set_error("dpa4c_model_info: null argument");
    return DPA4C_ERR_INVALID_ARG;
  }
  int64_t v[13] = {m->C0, m->L, m->R, m->S, m->D_out, m->F, m->n_layers, m->n_types,
                   m->n_rows, m->C[1], m->C[2], m->K[1], m->fold_allowed ? kFoldWords : 0};
  std::memcpy(info, v, sizeof(v));
  return 0;
}

int build_neighbors(const double* pos, int64_t N, const double cell[9], const int pbc[3],
                    double r_list, int64_t* row_ptr, int32_t* nbr_j, int32_t* nbr_shift,
                    int64_t cap, int64_t* n_pairs, void* stream) {
  if (!n_pairs || !row_ptr || N < 0 || cap < 0 || (N > 0 && !pos) || (cap > 0 && (!nbr_j || !nbr_shift))) {
    set_error("build_neighbors: bad pointer or size");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (N >= (int64_t(1) << 31)) {
    set_error("build_neighbors: at most 2^31 - 1 atoms");
    return DPA4C_ERR_INVALID_ARG;
  }
  CellSpec cs;
  int rc = cell_spec(cell, pbc, &cs);
  if (rc) return rc;
  if (!(r_list > 0.0) || !(r_list < 1000.0)) {
    set_error("build_neighbors: r_list must be in (0, 1000) A");
    return DPA4C_ERR_INVALID_ARG;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  DPA4C_HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(g_nb_lock);
  NeighborScratch*& nb = g_nb_scratch[dev];
  if (!nb) nb = new NeighborScratch();
  double ecell[9];
  rc = effective_cell(cs, pos, N, r_list, *nb, st, ecell);
  if (rc) return rc;
  CellGrid g;
  rc = make_grid(ecell, qfix_host(r_list), &g);
  if (rc) return rc;
  DevBuf*& fl = g_nb_flags[dev];
  if (!fl) fl = new DevBuf();
  DPA4C_TRY(fl->ensure(8 * 8));
  if (!nb->host_flag.p) {
    DPA4C_HIP_TRY(hipHostMalloc(&nb->host_flag.p, 64, hipHostMallocDefault));
    nb->host_flag.bytes = 64;
  }
  int64_t* hflag = nb->host_flag.as<int64_t>();
  if (N == 0) {
    DPA4C_HIP_TRY(hipMemsetAsync(row_ptr, 0, sizeof(int64_t), st));
    DPA4C_HIP_TRY(hipStreamSynchronize(st));
    *n_pairs = 0;
    return 0;
  }
  int64_t* flags = fl->as<int64_t>();
  DPA4C_HIP_TRY(hipMemsetAsync(flags, 0, 64, st));
  rc = build_skin_list(*nb, pos, N, g, row_ptr, flags, st);
  if (rc) return rc;
  DPA4C_HIP_TRY(hipMemcpyAsync(hflag, row_ptr + N, 8, hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipMemcpyAsync(hflag + 1, flags, 8, hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipMemcpyAsync(hflag + 2, flags + 3, 8, hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  if (hflag[1] & kFlagNonFinite) return flags_to_error(hflag[1]);
  *n_pairs = hflag[0];
  if (hflag[0] > cap) {
    set_error("build_neighbors: capacity " + std::to_string(cap) + " < " + std::to_string(hflag[0]) +
              " edges");
    return DPA4C_ERR_CAPACITY;
  }
  rc = fill_skin_list(*nb, N, g, row_ptr, nbr_j, nbr_shift, cap, flags, hflag[2], nullptr, st);
  if (rc) return rc;
  DPA4C_HIP_TRY(hipMemcpyAsync(hflag + 1, flags, 8, hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  return flags_to_error(hflag[1]);
}

}  // extern "C"

namespace dpa4c {

void eval_buf_sizes(int64_t n, int64_t cap, int ns, size_t sizes[kEvalBufs]) {
  const size_t nn = n < 1 ? 1 : size_t(n), cc = cap < 1 ? 1 : size_t(cap);
  auto r256 = [](size_t b) { return (b + 255) / 256 * 256; };
  const size_t raw[kEvalBufs] = {4 * nn,       16 * cc,      4 * cc,
                                 8 * cc,       4 * nn * size_t(ns),
                                 4 * nn * size_t(ns),        8 * (size_t(partial_count(int64_t(nn))) + 8),
                                 4 * nn,       4 * sizeof(uint32_t), 2 * sizeof(int64_t)};
  for (int k = 0; k < kEvalBufs; ++k) sizes[k] = r256(raw[k]);
}

// compute_energy_forces with the optional virial (virial == nullptr: none)
int energy_forces_core(const dpa4c_model* m, const double* pos, const int32_t* species, int64_t N,
                       const double cell[9], const int pbc[3], double r_c, const int64_t* row_ptr,
                       const int32_t* nbr_j, const int32_t* nbr_shift, int64_t n_pairs,
                       double* e_atom, double* forces, double* e_total, double* virial,
                       double* atom_virial, const EvalBufs* bufs, void* stream) {
  if (!m || N < 0 || n_pairs < 0 || !row_ptr || !e_total ||
      (N > 0 && (!pos || !species || !e_atom || !forces)) ||
      (n_pairs > 0 && (!nbr_j || !nbr_shift))) {
    set_error("compute_energy_forces: bad pointer or size");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (N >= (int64_t(1) << 31)) {
    set_error("compute_energy_forces: at most 2^31 - 1 atoms");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (std::fabs(r_c - m->r_c) > 1e-12) {
    set_error("compute_energy_forces: r_c differs from the model's cutoff");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (bufs && virial) {
    set_error("compute_energy_forces: no virial on caller-free buffers");
    return DPA4C_ERR_INVALID_ARG;
  }
  CellSpec cs;
  int rc = cell_spec(cell, pbc, &cs);
  if (rc) return rc;
  DeviceGuard guard(m->device);
  dpa4c_model* mm = const_cast<dpa4c_model*>(m);
  std::lock_guard<std::mutex> lock(mm->mu_lock);
  Workspace& w = mm->ws;
  hipStream_t st = static_cast<hipStream_t>(stream);
  double ecell[9];   // open axes: a placeholder length (compaction does not use it)
  rc = effective_cell(cs, nullptr, 0, m->r_c, w.nb, st, ecell);
  if (rc) return rc;
  CellGrid g;
  rc = make_grid(ecell, qfix_host(m->r_c), &g);
  if (rc) return rc;
  const bool own = bufs == nullptr;
  if (own) {
    rc = ensure_workspace(mm, N, n_pairs);
    if (rc) return rc;
  }
  const EvalBufs B = own ? ws_bufs(w) : *bufs;
  if (N == 0) {
    rc = launch_zero_i64(reinterpret_cast<int64_t*>(e_total), 1, st);
    if (rc == 0 && virial) rc = launch_zero_i64(reinterpret_cast<int64_t*>(virial), 9, st);
    return rc;
  }
  if (own) w.list_valid = false;   // the reverse index now describes the caller's list
  {
    StageScope t(m, kStSkinRev, st, own);
    // the reverse search's samples live in the edge records, which the
    // forward kernel rewrites before reading them
    rc = launch_zero_i64(B.check, 2, st);
    if (rc) return rc;
    rc = launch_skin_rev(row_ptr, nbr_j, nbr_shift, N, n_pairs, reinterpret_cast<int32_t*>(B.edge),
                         false, B.skin_rev, B.check, nullptr, st);
    if (rc) return rc;
  }
  // the list's size and the pairs found come back with the species mask
  // (prepare_species synchronises the stream)
  int64_t* hcheck = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(w.fold_host) + 16);
  DPA4C_HIP_TRY(hipMemcpyAsync(hcheck, row_ptr + N, sizeof(int64_t), hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipMemcpyAsync(hcheck + 1, B.check, sizeof(int64_t), hipMemcpyDeviceToHost, st));
  bool use_fold = false;
  rc = prepare_species(mm, species, N, B.fold_mask, B.fidx, own, &use_fold, st);
  if (rc) return rc;
  if (hcheck[0] > n_pairs || hcheck[0] < 0) {
    set_error("compute_energy_forces: the list holds row_ptr[N] = " + std::to_string(hcheck[0]) +
              " entries, outside [0, n_pairs = " + std::to_string(n_pairs) + "]");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (2 * hcheck[1] != hcheck[0]) {
    set_error("compute_energy_forces: the neighbour list is not symmetric (" +
              std::to_string(hcheck[0] - 2 * hcheck[1]) + " of " + std::to_string(hcheck[0]) +
              " entries have no reverse (j -> i, -n))");
    return DPA4C_ERR_INVALID_ARG;
  }
  VirialOut vo{};
  if (virial) {
    if (own) {
      DPA4C_TRY(w.virpart.ensure(2 * 9 * 8 * size_t(tail_partial_count(N))));
      if (!atom_virial) DPA4C_TRY(w.watom.ensure(9 * 8 * size_t(N)));
    }
    vo.part_v = w.virpart.as<double>();
    vo.atom = atom_virial ? atom_virial : w.watom.as<double>();
  }
  return run_model(m, pos, species, N, g, row_ptr, nbr_j, nbr_shift, n_pairs, B.skin_rev, e_atom,
                   forces, e_total, nullptr, virial ? &vo : nullptr, virial, B,
                   use_fold ? B.fidx : nullptr, own, st);
}

}  // namespace dpa4c

extern "C" {

int compute_energy_forces(const dpa4c_model* m, const double* pos, const int32_t* species,
                          int64_t N, const double cell[9], const int pbc[3], double r_c,
                          const int64_t* row_ptr, const int32_t* nbr_j, const int32_t* nbr_shift,
                          int64_t n_pairs, double* e_atom, double* forces, double* e_total,
                          void* stream) {
  return energy_forces_core(m, pos, species, N, cell, pbc, r_c, row_ptr, nbr_j, nbr_shift, n_pairs,
                            e_atom, forces, e_total, nullptr, nullptr, nullptr, stream);
}

int compute_energy_forces_virial(const dpa4c_model* m, const double* pos,
                                 const int32_t* species, int64_t N, const double cell[9],
                                 const int pbc[3], double r_c, const int64_t* row_ptr,
                                 const int32_t* nbr_j, const int32_t* nbr_shift, int64_t n_pairs,
                                 double* e_atom, double* forces, double* e_total, double* virial,
                                 double* atom_virial, void* stream) {
  if (!virial) {
    set_error("compute_energy_forces_virial: null virial");
    return DPA4C_ERR_INVALID_ARG;
  }
  return energy_forces_core(m, pos, species, N, cell, pbc, r_c, row_ptr, nbr_j, nbr_shift, n_pairs,
                            e_atom, forces, e_total, virial, atom_virial, nullptr, stream);
}

}  // extern "C"

namespace {

// Velocity-Verlet dynamics, NVE or (with ``nvt``) Nose-Hoover-chain NVT.
int dynamics(const dpa4c_model* m, double* pos, double* vel, const int32_t* species,
             const double* mass_by_species, int64_t N, const double cell[9], const int pbc[3],
             double r_c, double skin, double dt_fs, int nsteps, int rebuild_every, double* e_pot,
             double* e_kin, double* forces, int64_t* n_rebuilds, void* stream,
             const NvtConfig* nvt) {
  if (!m || N <= 0 || nsteps < 0 || !pos || !vel || !species || !mass_by_species || !forces ||
      (nsteps > 0 && (!e_pot || !e_kin))) {
    set_error(std::string(nvt ? "nvt_step: " : "verlet_step: ") + "bad pointer or size");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (N >= (int64_t(1) << 31)) {
    set_error(std::string(nvt ? "nvt_step: " : "verlet_step: ") + "at most 2^31 - 1 atoms");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (std::fabs(r_c - m->r_c) > 1e-12 || !(skin >= 0.0) || skin > 100.0 || !(dt_fs > 0.0) ||
      !(dt_fs < 100.0)) {
    set_error(std::string(nvt ? "nvt_step: " : "verlet_step: ") + "r_c must equal the model's; skin in [0, 100] A; dt in (0, 100) fs");
    return DPA4C_ERR_INVALID_ARG;
  }
  const int T1 = m->n_types + 1;
  for (int t = 0; t < T1; ++t)
    if (!(mass_by_species[t] > 0.0) || !std::isfinite(mass_by_species[t])) {
      set_error(std::string(nvt ? "nvt_step: " : "verlet_step: ") + "masses must be positive and finite");
      return DPA4C_ERR_INVALID_ARG;
    }
  CellSpec cs;
  int rc = cell_spec(cell, pbc, &cs);
  if (rc) return rc;
  DeviceGuard guard(m->device);
  dpa4c_model* mm = const_cast<dpa4c_model*>(m);
  std::lock_guard<std::mutex> lock(mm->mu_lock);
  Workspace& w = mm->ws;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t rcq = qfix_host(m->r_c), skq = qfix_host(skin);
  // the grids of the skin list and of the compaction; with open axes they
  // follow the extent of the atoms and are rebuilt with every list
  CellGrid g_list, g_cut;
  auto make_grids = [&]() -> int {
    double ec[9];
    int r = effective_cell(cs, cs.any_open ? pos : nullptr, N, m->r_c + skin, w.nb, st, ec);
    if (r) return r;
    r = make_grid(ec, rcq + skq, &g_list);
    if (r) return r;
    return make_grid(ec, rcq, &g_cut);
  };
  rc = make_grids();
  if (rc) return rc;

  // masses on the device
  const int np_tail = tail_partial_count(N);
  DPA4C_TRY(w.inv_mass.ensure(8 * T1));
  DPA4C_TRY(w.mass.ensure(8 * T1));
  DPA4C_TRY(w.flags.ensure(64));
  DPA4C_TRY(w.tailpart.ensure(32 * size_t(np_tail)));
  DPA4C_TRY(w.skin_row.ensure(8 * (N + 1)));
  DPA4C_TRY(w.qbuild.ensure(8 * 3 * N));
  if (!w.host_flags) DPA4C_HIP_TRY(hipHostMalloc((void**)&w.host_flags, 64, hipHostMallocDefault));
  {
    std::vector<double> im(T1);
    for (int t = 0; t < T1; ++t) im[t] = 1.0 / (mass_by_species[t] * (1.66053906660e-17 / 1.602176634e-19));
    DPA4C_HIP_TRY(hipMemcpyAsync(w.inv_mass.p, im.data(), 8 * T1, hipMemcpyHostToDevice, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(w.mass.p, mass_by_species, 8 * T1, hipMemcpyHostToDevice, st));
  }
  DPA4C_TRY(w.fidx.ensure(4 * size_t(N)));
  DPA4C_TRY(w.fold_mask.ensure(4 * sizeof(uint32_t)));
  bool use_fold = false;
  rc = prepare_species(mm, species, N, w.fold_mask.as<uint32_t>(), w.fidx.as<int32_t>(), true,
                       &use_fold, st);
  if (rc) return rc;
  const int32_t* fidx = use_fold ? w.fidx.as<int32_t>() : nullptr;
  int64_t* flags = w.flags.as<int64_t>();
  DPA4C_HIP_TRY(hipMemsetAsync(flags, 0, 64, st));

  // NVT: the chain state [xi, v, scale] (S words), its batch backup, the
  // kinetic partials of the current velocities and the virial partials
  NhcArgs nhc{};
  double* nvt_state = nullptr;
  double* nvt_backup = nullptr;
  double* kin_part = nullptr;
  const int npk = kinetic_partial_count(N);
  if (nvt) {
    const int M = nvt->length;
    const size_t S = 2 * size_t(M) + 1;
    DPA4C_TRY(w.nvt.ensure(8 * (2 * S + size_t(npk))));
    DPA4C_TRY(w.virpart.ensure(2 * 9 * 8 * size_t(np_tail)));
    DPA4C_TRY(w.watom.ensure(9 * 8 * size_t(N)));
    nvt_state = w.nvt.as<double>();
    nvt_backup = nvt_state + S;
    kin_part = nvt_backup + S;
    DPA4C_HIP_TRY(hipMemcpyAsync(nvt_state, nvt->chain, 16 * size_t(M), hipMemcpyDeviceToDevice, st));
    nhc.state = nvt_state;
    nhc.M = M;
    nhc.kT = 8.617333262e-5 * nvt->temperature;   // Boltzmann constant in eV/K (CODATA 2018)
    nhc.nf = double(3 * N - 3);
    nhc.dt = dt_fs;
    for (int k = 0; k < M; ++k)
      nhc.Q[k] = (k == 0 ? nhc.nf : 1.0) * nhc.kT * nvt->t_damp * nvt->t_damp;
  }
  auto vir_part = [&](int64_t s) { return w.virpart.as<double>() + (s & 1) * 9 * size_t(np_tail); };

  // a build of the skin list: count, read the size back, grow the capacity
  // if needed, fill, reverse index and the positions of the build
  auto initial_build = [&]() -> int {
    int r;
    w.list_valid = false;
    if (cs.any_open) {
      r = make_grids();
      if (r) return r;
    }
    {
      StageScope t(m, kStNeighbor, st);
      r = build_skin_list(w.nb, pos, N, g_list, w.skin_row.as<int64_t>(), flags, st);
      if (r) return r;
    }
    DPA4C_HIP_TRY(hipMemcpyAsync(w.host_flags, w.skin_row.as<int64_t>() + N, 8,
                                 hipMemcpyDeviceToHost, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(w.host_flags + 1, flags, 8, hipMemcpyDeviceToHost, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(w.host_flags + 2, flags + 3, 8, hipMemcpyDeviceToHost, st));
    DPA4C_HIP_TRY(hipStreamSynchronize(st));
    if (w.host_flags[1]) return flags_to_error(w.host_flags[1]);
    const int64_t need = w.host_flags[0];
    if (need > w.cap || !w.skin_j.p) {
      // 1/8 headroom over the need (plus 16 per atom) before the next
      // reallocation; the per-edge workspace is sized with it
      const int64_t cap = need + need / 8 + 16 * N;
      DPA4C_TRY(w.skin_j.ensure(4 * size_t(cap)));
      DPA4C_TRY(w.skin_shift.ensure(4 * size_t(cap)));
      w.cap = cap;
    }
    r = ensure_workspace(mm, N, w.cap);
    if (r) return r;
    StageScope t(m, kStNeighbor, st);
    // the samples for the reverse search go to the edge records, which the
    // forward kernel rewrites before reading them
    r = fill_skin_list(w.nb, N, g_list, w.skin_row.as<int64_t>(), w.skin_j.as<int32_t>(),
                       w.skin_shift.as<int32_t>(), w.cap, flags, w.host_flags[2],
                       w.edge.as<int32_t>(), st);
    if (r) return r;
    r = launch_skin_rev(w.skin_row.as<int64_t>(), w.skin_j.as<int32_t>(), w.skin_shift.as<int32_t>(),
                        N, w.cap, w.edge.as<int32_t>(), true, w.skin_rev.as<int64_t>(), nullptr,
                        &w.nb, st);
    if (r) return r;
    r = launch_snapshot_q(pos, N, w.qbuild.as<int64_t>(), st);
    if (r) return r;
    // open axes: the grid follows the atoms, so the list is not carried over
    w.list_valid = !cs.any_open;
    w.list_n = N;
    w.list_rq = rcq + skq;
    for (int k = 0; k < 9; ++k) w.list_cell[k] = cs.cell[k];
    return 0;
  };
  // a displacement-triggered call whose list is still the one of the last
  // call starts with the displacement check instead of a build: any valid
  // list gives the same edges in the same order, so the trajectory does not
  // depend on it
  bool reuse = rebuild_every == 0 && w.list_valid && w.list_n == N && w.list_rq == rcq + skq &&
               !cs.any_open;
  for (int k = 0; reuse && k < 9; ++k) reuse = w.list_cell[k] == cs.cell[k];

  int64_t rebuilds = 0;
  // energy partials of step s in buffer s % 2, so that a step can add up
  // those of the step before while writing its own
  auto part_e = [&](int64_t s) { return w.tailpart.as<double>() + (s & 1) * 2 * size_t(np_tail); };
  auto sums_of = [&](int64_t s) {
    return s < 0 ? StepSums{nullptr, nullptr, 0, nullptr, nullptr}
                 : StepSums{part_e(s), part_e(s) + np_tail, np_tail, e_pot + s, e_kin + s};
  };
  // One step: kick/drift (unless ``kicked``: the force assembly of the step
  // before did it), with the displacement check against the last build when
  // ``check``; an optional rebuild; the model, whose force assembly also
  // does the second half kick, the energy partials of the step, the totals
  // of step ``prev`` and, with ``kick_next``, the kick and drift of the next
  // step (checked when ``check``).
  // NVT: the chain launch before a kick closes step ``prev`` (when >= 0) and
  // opens the next step
  auto chain_launch = [&](int64_t prev, bool open) -> int {
    NhcArgs a = nhc;
    if (prev >= 0) {
      a.part_k = part_e(prev) + np_tail;
      a.part_e = part_e(prev);
      a.part_v = vir_part(prev);
      a.np = np_tail;
      a.close_prev = 1;
      a.e_pot = e_pot + prev;
      a.e_kin = e_kin + prev;
      a.e_thermo = nvt->e_thermo + prev;
      a.virial = nvt->virial ? nvt->virial + 9 * prev : nullptr;
    } else {
      int r = launch_kinetic(vel, species, w.mass.as<double>(), T1, N, kin_part, st);
      if (r) return r;
      a.part_k = kin_part;
      a.np = npk;
    }
    a.open_next = open ? 1 : 0;
    return launch_nhc(a, st);
  };
  auto one_step = [&](int64_t step, bool check, bool rebuild, int64_t prev, bool kicked,
                      bool kick_next) -> int {
    if (nvt) {
      kicked = false;
      kick_next = false;
    }
    if (!kicked) {
      StageScope t(m, kStIntegrate, st);
      if (nvt) {
        // every step boundary as at the end of a batch or a call: the
        // closing half step and its velocity scale, then the opening half
        // step from the kinetic energy of the scaled velocities, so that a
        // run gives the same bits however it is split into batches and calls
        if (prev >= 0) {
          int r = chain_launch(prev, false);
          if (r) return r;
          r = launch_scale(vel, N, nvt_state + 2 * nvt->length, st);
          if (r) return r;
        }
        int r = chain_launch(-1, true);
        if (r) return r;
      }
      int r = launch_kick_drift(pos, vel, forces, species, w.inv_mass.as<double>(), T1, N, dt_fs,
                                1, check ? w.qbuild.as<int64_t>() : nullptr, skq, flags,
                                sums_of(-1), step, nvt ? nvt_state + 2 * nvt->length : nullptr,
                                st);
      if (r) return r;
    }
    if (rebuild) {
      int r = initial_build();
      if (r) return r;
      ++rebuilds;
    }
    // (NVT: the chain launch adds the step's partials up, not the force assembly)
    const StepTail tail{pos, vel, species, w.inv_mass.as<double>(), w.mass.as<double>(), T1,
                        0.5 * dt_fs, dt_fs, w.eatom.as<double>(), part_e(step),
                        part_e(step) + np_tail, nvt ? sums_of(-1) : sums_of(prev),
                        kick_next ? 1 : 0, check ? w.qbuild.as<int64_t>() : nullptr, skq, flags,
                        step + 1};
    VirialOut vo{};
    vo.part_v = nvt ? vir_part(step) : nullptr;
    vo.atom = w.watom.as<double>();
    return run_model(m, pos, species, N, g_cut, w.skin_row.as<int64_t>(),
                     w.skin_j.as<int32_t>(), w.skin_shift.as<int32_t>(), w.cap,
                     w.skin_rev.as<int64_t>(), w.eatom.as<double>(), forces, nullptr, &tail,
                     nvt ? &vo : nullptr, nullptr, ws_bufs(w), fidx, true, st);
  };
  // the end of a batch: the totals of step ``last`` (NVT: its closing chain
  // half step and velocity scaling)
  auto finish = [&](int64_t last) -> int {
    StageScope t(m, kStIntegrate, st);
    if (nvt) {
      int r = chain_launch(last, false);
      if (r) return r;
      return launch_scale(vel, N, nvt_state + 2 * nvt->length, st);
    }
    return launch_final_step(sums_of(last), st);
  };
  const size_t nvt_words = nvt ? 2 * size_t(nvt->length) + 1 : 0;

  // Step 0 builds the list.  Later steps run in speculative batches without
  // rebuild checks on the host: kick/drift records the first step whose
  // displacement exceeds half the skin.  A batch without one stands; after
  // one at step v the state saved at the start of the batch is restored,
  // steps before v are replayed (bit-identical) and step v rebuilds the
  // list, exactly as a per-step check would.  Forced rebuilds
  // (rebuild_every > 0) start batches of their own.
  if (nsteps > 0 && !reuse) {
    rc = one_step(0, false, true, -1, false, false);
    if (rc) return rc;
    rc = finish(0);
    if (rc) return rc;
  }
  DPA4C_TRY(w.backup.ensure(3 * 24 * size_t(N)));
  double* bk = w.backup.as<double>();
  const size_t state = 24 * size_t(N);
  const double half_skin = 0.5 * skin;
  // step index of the last build (a carried-over list was built that many
  // steps before this call's first)
  int64_t last_build = reuse ? -1 - w.list_steps_since_build : 0, batch = 8;
  double growth = 0.0;   // A per step since the last build, from the last batch
  for (int64_t s = reuse ? 0 : 1; s < nsteps;) {
    if (rebuild_every > 0 && s % rebuild_every == 0) {
      rc = one_step(s, true, true, -1, false, false);
      if (rc) return rc;
      rc = finish(s);
      if (rc) return rc;
      last_build = s++;
      continue;
    }
    int64_t e = s + batch < nsteps ? s + batch : nsteps;
    if (rebuild_every > 0) {
      const int64_t next_forced = (s / rebuild_every + 1) * rebuild_every;
      if (next_forced < e) e = next_forced;
    }
    DPA4C_HIP_TRY(hipMemcpyAsync(bk, pos, state, hipMemcpyDeviceToDevice, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(bk + 3 * N, vel, state, hipMemcpyDeviceToDevice, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(bk + 6 * N, forces, state, hipMemcpyDeviceToDevice, st));
    if (nvt)
      DPA4C_HIP_TRY(hipMemcpyAsync(nvt_backup, nvt_state, 8 * nvt_words, hipMemcpyDeviceToDevice, st));
    rc = launch_set_flag(flags, 4, INT64_MAX, st);
    if (rc) return rc;
    rc = launch_set_flag(flags, 5, 0, st);
    if (rc) return rc;
    for (int64_t t = s; t < e; ++t) {
      rc = one_step(t, true, false, t > s ? t - 1 : -1, t > s, t + 1 < e);
      if (rc) return rc;
    }
    rc = finish(e - 1);
    if (rc) return rc;
    DPA4C_HIP_TRY(hipMemcpyAsync(w.host_flags, flags, 64, hipMemcpyDeviceToHost, st));
    DPA4C_HIP_TRY(hipStreamSynchronize(st));
    rc = flags_to_error(w.host_flags[0]);
    if (rc) return rc;
    const int64_t v = w.host_flags[4];
    if (v == INT64_MAX) {
      // no violation: size the next batch from the displacement growth
      const double d = std::sqrt(double(w.host_flags[5])) / kQScale;
      growth = d / double(e - last_build);
      const double left = growth > 0.0 ? (half_skin - d) / growth : 64.0;
      batch = static_cast<int64_t>(0.75 * left);
      batch = batch < 1 ? 1 : (batch > 64 ? 64 : batch);
      s = e;
      continue;
    }
    if (rebuild_every < 0) {
      set_error(std::string(nvt ? "nvt_step: " : "verlet_step: ") + "an atom moved more than skin/2 and rebuilds are disabled");
      return DPA4C_ERR_SKIN;
    }
    // violation at step v: the displacement reached half the skin within
    // v - last_build steps, a growth rate for sizing the batches that follow
    const double g_viol = half_skin / double(v - last_build > 0 ? v - last_build : 1);
    growth = growth > g_viol ? growth : g_viol;
    // restore, replay [s, v), rebuild at v
    DPA4C_HIP_TRY(hipMemcpyAsync(pos, bk, state, hipMemcpyDeviceToDevice, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(vel, bk + 3 * N, state, hipMemcpyDeviceToDevice, st));
    DPA4C_HIP_TRY(hipMemcpyAsync(forces, bk + 6 * N, state, hipMemcpyDeviceToDevice, st));
    if (nvt)
      DPA4C_HIP_TRY(hipMemcpyAsync(nvt_state, nvt_backup, 8 * nvt_words, hipMemcpyDeviceToDevice, st));
    for (int64_t t = s; t < v; ++t) {
      rc = one_step(t, false, false, t > s ? t - 1 : -1, t > s, t + 1 < v);
      if (rc) return rc;
    }
    if (v > s) {
      rc = finish(v - 1);
      if (rc) return rc;
    }
    rc = one_step(v, false, true, -1, false, false);
    if (rc) return rc;
    rc = finish(v);
    if (rc) return rc;
    last_build = v;
    s = v + 1;
    batch = static_cast<int64_t>(0.75 * half_skin / growth);
    batch = batch < 1 ? 1 : (batch > 64 ? 64 : batch);
  }
  if (nvt)
    DPA4C_HIP_TRY(hipMemcpyAsync(nvt->chain, nvt_state, 16 * size_t(nvt->length),
                                 hipMemcpyDeviceToDevice, st));
  DPA4C_HIP_TRY(hipMemcpyAsync(w.host_flags, flags, 64, hipMemcpyDeviceToHost, st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  if (n_rebuilds) *n_rebuilds = rebuilds;
  if (nsteps > 0) w.list_steps_since_build = nsteps - 1 - last_build;
  return flags_to_error(w.host_flags[0]);
}

}  // namespace

extern "C" {

int verlet_step(const dpa4c_model* m, double* pos, double* vel, const int32_t* species,
                const double* mass_by_species, int64_t N, const double cell[9], const int pbc[3],
                double r_c, double skin, double dt_fs, int nsteps, int rebuild_every,
                double* e_pot, double* e_kin, double* forces, int64_t* n_rebuilds, void* stream) {
  return dynamics(m, pos, vel, species, mass_by_species, N, cell, pbc, r_c, skin, dt_fs, nsteps,
                  rebuild_every, e_pot, e_kin, forces, n_rebuilds, stream, nullptr);
}

int nvt_step(const dpa4c_model* m, double* pos, double* vel, const int32_t* species,
             const double* mass_by_species, int64_t N, const double cell[9], const int pbc[3],
             double r_c, double skin, double dt_fs, int nsteps, int rebuild_every,
             double temperature, double t_damp_fs, int chain_length, double* chain, double* e_pot,
             double* e_kin, double* e_thermo, double* virial, double* forces,
             int64_t* n_rebuilds, void* stream) {
  if (!(temperature > 0.0) || !std::isfinite(temperature) || !(t_damp_fs > 0.0) ||
      !std::isfinite(t_damp_fs) || chain_length < 1 || chain_length > kMaxChain || !chain ||
      (nsteps > 0 && !e_thermo) || N < 2) {
    set_error("nvt_step: temperature and damping time must be positive, chain length in [1, 8], "
              "chain and e_thermo given, N >= 2");
    return DPA4C_ERR_INVALID_ARG;
  }
  const NvtConfig cfg{temperature, t_damp_fs, chain_length, chain, e_thermo, virial};
  return dynamics(m, pos, vel, species, mass_by_species, N, cell, pbc, r_c, skin, dt_fs, nsteps,
                  rebuild_every, e_pot, e_kin, forces, n_rebuilds, stream, &cfg);
}

int dpa4c_debug_stages(const dpa4c_model* m, int64_t N, float* node_state, float* descriptor,
                       int32_t* edge_count, void* stream) {
  if (!m || N < 0 || N != m->last_n || !m->ws.last_species) {
    set_error("dpa4c_debug_stages: N must match the last evaluation on this model");
    return DPA4C_ERR_INVALID_ARG;
  }
  DeviceGuard guard(m->device);
  dpa4c_model* mm = const_cast<dpa4c_model*>(m);
  std::lock_guard<std::mutex> lock(mm->mu_lock);
  Workspace& w = mm->ws;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (N == 0) return 0;
  // recompute node state and descriptor from the stored compacted edges
  const CompactArgs ca = compact_args(w.last_grid, w.last_pos, w.skin_j_used, w.skin_shift_used,
                                      qfix_host(m->r_c), w.cap_used, ws_bufs(w));
  int rc = launch_forward(m, N, w.last_species, w.last_fidx, w.skin_row_used, ca,
                          w.node.as<float>(), st);
  if (rc) return rc;
  DPA4C_TRY(w.desc.ensure(size_t(4) * N * m->D_out));
  DPA4C_TRY(w.eatom.ensure(size_t(8) * N));
  rc = launch_atoms(m, N, w.last_species, w.node.as<float>(), w.node_grad.as<float>(),
                    w.eatom.as<double>(), w.desc.as<float>(), st);
  if (rc) return rc;
  if (node_state)
    DPA4C_HIP_TRY(hipMemcpyAsync(node_state, w.node.p, 4 * N * (m->S + 2), hipMemcpyDeviceToDevice, st));
  if (descriptor)
    DPA4C_HIP_TRY(hipMemcpyAsync(descriptor, w.desc.p, size_t(4) * N * m->D_out,
                                 hipMemcpyDeviceToDevice, st));
  if (edge_count)
    DPA4C_HIP_TRY(hipMemcpyAsync(edge_count, w.ecount.p, 4 * N, hipMemcpyDeviceToDevice, st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  return 0;
}

int dpa4c_set_timing(dpa4c_model* m, int64_t stage_mask) {
  if (!m) {
    set_error("dpa4c_set_timing: null model");
    return DPA4C_ERR_INVALID_ARG;
  }
  DeviceGuard guard(m->device);
  collect_timing(m);
  m->timing.mask = stage_mask;
  return 0;
}

int dpa4c_get_timings(dpa4c_model* m, double* ms, int64_t* count, int n) {
  if (!m || n < 0) {
    set_error("dpa4c_get_timings: bad argument");
    return DPA4C_ERR_INVALID_ARG;
  }
  DeviceGuard guard(m->device);
  collect_timing(m);
  for (int s = 0; s < n && s < kNumStages; ++s) {
    if (ms) ms[s] = m->timing.ms[s];
    if (count) count[s] = m->timing.count[s];
    m->timing.ms[s] = 0;
    m->timing.count[s] = 0;
  }
  return kNumStages;
}

const char* dpa4c_stage_name(int s) { return stage_name(s); }

int dpa4c_debug_gemm(const float* A, const float* B, float* C, int M, int N, int K, void* stream) {
  if (!A || !B || !C || M < 0 || N <= 0 || N % 4 || K <= 0 || K % 16) {
    set_error("dpa4c_debug_gemm: need K % 16 == 0 and N % 4 == 0");
    return DPA4C_ERR_INVALID_ARG;
  }
  return launch_gemm_test(A, B, C, M, N, K, static_cast<hipStream_t>(stream));
}

const char* dpa4c_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
