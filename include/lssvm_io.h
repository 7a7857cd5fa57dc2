/*
 * lssvm_io.h - host-side file IO around the LS-SVM training path.
 *
 * The paper's training pipeline reads the whole training set from a file,
 * converts sparse input to dense by filling in zeros, solves, and writes the
 * learned support vectors and weights to a model file (Sec. III, the four
 * steps of training; Sec. IV-E times them as read / transform / cg / write).
 * Its files follow LIBSVM's text formats, and these functions read and write
 * the same formats.
 *
 * Data file: one point per line, "<label> <index>:<value> <index>:<value> ...",
 * indices 1-based and strictly increasing; absent features are 0. Blank lines
 * are skipped. Values are parsed as correctly rounded doubles and then
 * rounded to the requested dtype.
 *
 * Model file: a header of "key value" lines (svm_type, kernel_type, degree,
 * gamma, coef0, nr_class, total_sv, rho, label, nr_sv), then "SV" and one line
 * per support vector "<coef> <index>:<value> ...". For the LS-SVM every point
 * is a support vector with coef = alpha_i, grouped label +1 first, and
 * rho = -b, so that coef-weighted kernel values minus rho is the decision
 * value f(x) = sum_i alpha_i k(x_i, x) + b.
 *
 * All pointers are HOST pointers owned by the caller. dtype is LSSVM_F64 or
 * LSSVM_F32 (lssvm.h). num_threads <= 0 uses every hardware thread. Return
 * values are the status codes of lssvm.h (LSSVM_EINVAL for bad arguments,
 * unreadable files and malformed lines, with the line number in
 * lssvm_last_error()). These calls do no GPU work.
 */
#ifndef LSSVM_IO_H_
#define LSSVM_IO_H_

#include <stddef.h>
#include <stdint.h>

#include "lssvm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Count the points (non-blank lines) of a data file and its largest feature
 * index (= the dense dimension d; 0 if no line has a feature). */
int lssvm_libsvm_scan(const char* path, int64_t* n_out, int64_t* d_out, int32_t num_threads);

/* Read a data file into X (n x d row-major, dtype, zero-filled where a
 * feature is absent) and y (n, dtype). n and d must be those lssvm_libsvm_scan
 * reported (a larger d is allowed and zero-padded). */
int lssvm_libsvm_read(const char* path, int32_t dtype, void* X, void* y, int64_t n, int64_t d,
                      int32_t num_threads);

/* Write n points of d features (X row-major, y labels, dtype) as a data file;
 * zero features are omitted. Values are written in the shortest form that
 * reads back to the same value. */
int lssvm_libsvm_write(const char* path, int32_t dtype, const void* X, const void* y, int64_t n,
                       int64_t d, int32_t num_threads);

/* Write the trained model: kernel and parameters, rho = -b, and every point
 * (X, y, alpha: n x d, n, n, dtype) as a support vector, label +1 first. */
int lssvm_model_write(const char* path, int32_t dtype, int32_t kernel, const lssvm_params* kp,
                      double b, const void* alpha, const void* X, const void* y, int64_t n,
                      int64_t d, int32_t num_threads);

/* Read a model header: kernel, parameters, b (= -rho), number of support
 * vectors n and largest feature index d. */
int lssvm_model_scan(const char* path, int32_t* kernel, lssvm_params* kp, double* b,
                     int64_t* n_out, int64_t* d_out);

/* Read the support vectors of a model: X (n x d row-major), alpha and the
 * labels y (+1 for the first nr_sv[0] vectors, -1 after), all dtype. */
int lssvm_model_read(const char* path, int32_t dtype, void* X, void* alpha, void* y, int64_t n,
                     int64_t d, int32_t num_threads);

#ifdef __cplusplus
}
#endif

#endif /* LSSVM_IO_H_ */
