"""fp64 CPU oracle for the BitsMoE spectral quantizer hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import or call anything here.
The product path (``paper_2606_00079_amd``) never imports this package and
shares no code with it; the oracle in turn never imports the product.

Each function is a plain, slow, obviously correct numpy implementation of a
definition from the paper (arXiv 2606.00079, "BitsMoE"), in fp64:

* ``gram``           H = X Diag(g) X^T with g_t = 1/n       (App. B.2, Eq. app_affinity_gram)
* ``gram_experts``   M = W_cat W_cat^T = sum_e W_e W_e^T       (App. B.1, Eqs. app_down_w_cat,
                                                               app_down_cat_svd_absorbed)
* ``shared_basis``   top-r eigenvectors of M = left singular vectors of W_cat
* ``project``        C_e = U^T W_e  (spectral factors, P~_e^T of Eq. app_down_p_tilde_partition)
* ``quant_group``    group-wise asymmetric min/max round-to-nearest quantizer
* ``score``          L[u, b] = delta H delta^T, delta = c - Q_b(c)  (App. B.2, Eq. app_down_exact_metric)
* ``allocate_dp``    exact multiple-choice knapsack, one per projection (Sec. 3.3,
                     Eq. ilp_piecewise_projection; App. B.4, Eq. ilp_piecewise_eps)
* ``pack``/``unpack`` bit-plane packing of the chosen codes
* ``inspace``        the input-space basis of gate/up (Sec. 3.2): M_in = sum W_e^T W_e,
                     units W_e phi_k, beta_k = phi_k^T H phi_k and the diagonal-approximation
                     loss beta_k ||c - Q_b(c)||^2
* ``routed``         routing-affinity-weighted calibration Grams H_e per expert
                     (App. B.2, Eq. app_affinity_gram) and their loss table
* ``decode``         stage-3 inference from the packed factors: y = U sum_j g_j C^_e x
                     (output space) and y = sum_j g_j C^_e^T Phi^T x (input space)
                     (Sec. 4.4)
* ``surrogate``      the paper's piecewise surrogate cost alpha^2 beta^gamma E(b) over the
                     widths {0,1,2,3,4,6,8,16}, its quantizers and the equivalent-bit
                     budget (App. B.3-B.5, Theorem app_spectrum_loss)

Readings where the paper is silent are stated in each function.  Every
function here is pinned by CPU tests against closed forms, brute force or
independent library routines (``tests/test_oracle_*.py``).
"""
from .spectral import gram, gram_experts, shared_basis, project, unit_energy, truncation_loss
from .quant import (quant_group, fake_quant, score, score_rows, pack_layout, pack, unpack,
                    bit_planes)
from .ilp import integerize, allocate_dp, allocate_exhaustive, objective
from . import surrogate, inspace, routed, decode
from .surrogate import surrogate_table, budget_equivalent

__all__ = [
    "gram", "gram_experts", "shared_basis", "project", "unit_energy", "truncation_loss",
    "quant_group", "fake_quant", "score", "score_rows", "pack_layout", "pack", "unpack",
    "bit_planes", "integerize", "allocate_dp", "allocate_exhaustive", "objective",
    "surrogate", "surrogate_table", "budget_equivalent", "inspace", "routed", "decode",
]
