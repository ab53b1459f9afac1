"""NestQuant oracle: a plain, slow, CPU-only fp64/exact implementation of the method.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP kernels, the C ABI
library or its Python binding) may import, call, link or execute anything in this
package.  Only the tests, the smoke check and the CPU-baseline leg of the benchmark
use it, to check and to time the GPU path against the paper's definitions.

It shares no code with the GPU path.  It is written from the paper
(NestQuant, arXiv 2502.09720):

* ``lattice``   -- the Gosset lattice E8 (Sec. 3 "Lattices", App. C Alg. 5 "Oracle for
                   the Gosset lattice") and the generator G of 2E8 (App. E);
* ``voronoi``   -- Voronoi code encode / decode (Sec. 4.1, Alg. 1 and Alg. 2);
* ``nestquant`` -- the row quantizer (Sec. 4.2, Alg. 3) with the First-beta and Opt-beta
                   strategies (App. F), decoding, the dot product of two coded vectors
                   (Alg. 4) and the coded matrix product built from it;
* ``layout``    -- the packed storage of codes, beta indices and scales;
* ``theory``    -- closed forms the paper states (rate, Gamma(R) bound, NSM of E8);
* ``rotation``  -- the Hadamard rotation of rows (Sec. 5);
* ``beta_dp``   -- the choice of the beta set (App. F, Alg. 6) and the synthetic
                   rate-distortion frontier (Sec. 6.1).

Every function that the paper does not fix completely states the reading it takes.
"""

from . import lattice, voronoi, nestquant, layout, theory, rotation, beta_dp  # noqa: F401
