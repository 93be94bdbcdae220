// Test driver for the PCA fit's host linear algebra (csrc/host_linalg.hpp): reads
// "chol n a00 a01 ...", "cholr n ..." (a pivot threshold of 1e-9 of the largest diagonal) or
// "eig n a00 a01 ..." (row-major) on stdin and prints the result: chol / cholr -> "ok" and
// R^{-1} (row-major) or "notpd"; eig -> the eigenvalues, then V^T (row-major), or
// "notconverged"; eigcap -> the same solve allowed one QR step: "converged" or "notconverged".
#include <stdio.h>
#include <string.h>

#include "host_linalg.hpp"

int main() {
  char mode[8];
  int n;
  if (scanf("%7s %d", mode, &n) != 2) return 2;
  std::vector<double> A((size_t)n * n);
  for (double& x : A)
    if (scanf("%lf", &x) != 1) return 2;
  if (strcmp(mode, "chol") == 0 || strcmp(mode, "cholr") == 0) {
    std::vector<double> Ri;
    if (!hmoe::chol_inverse(A, n, Ri, strcmp(mode, "cholr") == 0 ? 1e-9 : 0.0)) {
      printf("notpd\n");
      return 0;
    }
    printf("ok\n");
    for (double x : Ri) printf("%.17g\n", x);
  } else if (strcmp(mode, "eigcap") == 0) {  // one QR step at most: must report non-convergence
    std::vector<double> w, VT;
    printf("%s\n", hmoe::sym_eigen(A, n, w, VT, 1) ? "converged" : "notconverged");
  } else {
    std::vector<double> w, VT;
    if (!hmoe::sym_eigen(A, n, w, VT)) {
      printf("notconverged\n");
      return 0;
    }
    for (double x : w) printf("%.17g\n", x);
    for (double x : VT) printf("%.17g\n", x);
  }
  return 0;
}
