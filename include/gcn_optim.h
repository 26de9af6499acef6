/*
 * gcn_optim.h -- the optimiser step of graph-sampling GCN training: Alg. 1
 * (arXiv 1810.11899) updates the weights with ADAM after each backward pass.
 *
 * Conventions are those of gcn_layer.h (device pointers owned by the caller,
 * `stream` a hipStream_t as void*, host checks before any launch, negative
 * gcn_status on failure with a message for gcn_last_error()).
 */
#ifndef GCN_OPTIM_H_
#define GCN_OPTIM_H_

#include <stdint.h>

#include "gcn_layer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One Adam step (Kingma and Ba, ICLR 2015, Algorithm 1) over `count` float32
 * parameters, in place, elementwise:
 *     m <- beta1 m + (1 - beta1) g;   v <- beta2 v + (1 - beta2) g^2
 *     p <- p - lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * params, m, v [count] are updated; grads [count] is read.  step counts from 1
 * (m and v start at zero before step 1).  The caller keeps every trained
 * tensor (weights, biases, prediction layer) in one flat buffer so that one
 * call updates them all.  The hyperparameters are host doubles; the
 * coefficients 1 - beta, lr / (1 - beta1^step) and 1 / sqrt(1 - beta2^step)
 * are formed in double and rounded once to float32. */
int gcn_adam_update(float *params, const float *grads, float *m, float *v, int64_t count, double lr,
                    double beta1, double beta2, double eps, int32_t step, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GCN_OPTIM_H_ */
