"""CPU oracle for the diffusion-map kernel path -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, float64 statement of what the HIP path
computes.  Only the tests, the smoke check and the benchmark's CPU-baseline
leg may import it; the library and its Python binding never do, and this
package imports nothing from them.

Modules
-------
``kernel``      Gaussian affinity K = exp(-beta H) with H the pairwise squared
                distances written in difference form (Sec. 2.1, eq. kernel),
                and the scaled products diag(sl) K diag(sr) V
                (Sec. 2.1 eq. matmat, Sec. 2.2 eq. tiled_rbf), dense or on a
                subset of rows.
``normalise``   Coifman-Lafon alpha-normalisation: q, q^-alpha, d, s, the
                symmetric operator M and the Markov operator P
                (Sec. 2.1, eq. symmetric).
``eig``         dense LAPACK eigensolve of M, Markov eigenvectors
                (Sec. 2.3 first paragraph; last paragraph of Sec. 2.3).
``nystrom``     out-of-sample extension of Markov eigenvectors (Sec. 1, 2.3).
``torus_grid``  closed-form spectrum of the kernel on a regular grid of a
                flat torus (Kronecker product of circulants).
``diagnostics`` off-diagonal mass, Perron gap and precision wall
                (Sec. 2.3 eqs. neff, vmach, perronwall), principal angles.

Every function works in float64 on the values exactly as handed to it.
"""
