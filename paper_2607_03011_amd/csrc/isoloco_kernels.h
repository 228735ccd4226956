// Launch interface between the host planner and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>

#include "isoloco_types.h"

namespace isoloco {

// Device tables and buffers inside the caller's workspace, plus the host copies
// of the few values the launchers need to size grids.
struct DevTables {
  const MatInfo* mats;
  const Chunk* chunks;  // ISO chunks first, then AVG chunks
  const Task* gram_tasks;
  const Task* poly_tasks;
  const Task* update_tasks;
  MatScalars* scalars;
  double* part_sq;
  double* part_tr;
  float* delta;
  float* x[2];
  float* gram;
  float* poly;
  float* gpart;
  int n_mat, n_chunks, n_iso_chunks;
  int n_gram_tasks, n_poly_tasks, n_update_tasks;
  int n_split;
  const int* split_mats_host;  // host arrays of length n_split
  const int* split_n_host;
};

struct StepArgs {
  float* theta;
  float* mom;
  WorkerPtrs workers;
  int K;
  int worker_dtype;  // 0 float32, 1 bfloat16
  float alpha, lr, mu;
};

struct PolarStep {
  const float* xin;
  float* xout;
  float ca, cb, cc;
  int first;
};

hipError_t launch_reduce(const DevTables& t, const StepArgs& a, hipStream_t st);
hipError_t launch_fro(const DevTables& t, hipStream_t st);
// mode: 0 Gram, 1 polynomial, 2 update
hipError_t launch_gemm(const DevTables& t, int mode, const PolarStep& p, hipStream_t st);
hipError_t launch_split_sums(const DevTables& t, hipStream_t st);
// mode 0: normalisation of the first step; mode 1: orthonormality residual
hipError_t launch_gram_norm(const DevTables& t, int mode, int steps, hipStream_t st);
hipError_t launch_trace(const DevTables& t, const float* q, hipStream_t st);
hipError_t launch_finish(const DevTables& t, const float* q, const StepArgs& a, hipStream_t st);

}  // namespace isoloco
