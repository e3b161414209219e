"""MI355X-native Hessian-free curvature path (paper arXiv 1606.00511)."""
