"""fp64 CPU oracle (test infrastructure; never called by the library)."""
from .krpe_oracle import (prf_features, trf_features, elu_features, features, toeplitz_matrix,
                          toeplitz_product, toeplitz_rows, attention, attention_rows, attention_grad, normalize_rows)

__all__ = ["prf_features", "trf_features", "elu_features", "features", "toeplitz_matrix",
           "toeplitz_product", "toeplitz_rows", "attention", "attention_rows", "attention_grad", "normalize_rows"]
