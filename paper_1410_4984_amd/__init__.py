"""RBF-ARD psi-statistics and their gradients on MI355X (HIP, gfx950)."""
