"""Closed-loop driver on one GPU: Algorithm 2 (arXiv:2010.13359) on the
bilinear game min_x max_y x^T A y, the textbook min-max problem on which
plain gradient steps cycle outward (Section 2.2) while the optimistic method
converges.

Each worker m evaluates a noisy gradient F(w^{(m)}_{t-1/2}) + xi at its own
evaluation point -- the WX row the previous iteration produced -- with
F(x, y) = (A y, -A^T x) (the game's operator, the role of the GAN's
gradients); the library then runs the iteration (EF accumulate, compress,
aggregate, OMD update, next evaluation points).  The gradient oracle is a
torch matmul: it is the input of the compression path, not part of it.
"""
import torch

from . import dqgan


class BilinearGame:
    def __init__(self, n, seed=0, device="cuda"):
        self.n, self.d = n, 2 * n
        gen = torch.Generator(device="cpu").manual_seed(seed)
        self.A = (torch.randn(n, n, generator=gen) / n ** 0.5).to(device)

    def operator(self, Z):
        """F applied to every row of Z ([rows][>= 2n]); returns [rows][2n]."""
        x, y = Z[:, :self.n], Z[:, self.n:self.d]
        return torch.cat([y @ self.A.T, -(x @ self.A)], dim=1)


def run_bilinear(kind, n=512, M=4, T=800, eta=0.2, noise=0.05, seed=0, record_every=100, on_step=None,
                 **plan_kwargs):
    """Run T iterations; returns the list of ||w_t|| / ||w_0|| every
    `record_every` iterations.  `on_step(t, state)` (optional) is called
    before iteration t with the device state (G, E, W) of that iteration."""
    dev = torch.device("cuda")
    game = BilinearGame(n, seed, dev)
    plan = dqgan.Plan(game.d, M, kind, seed=seed + 1, **plan_kwargs)
    ld = plan.ld
    gen = torch.Generator(device=dev).manual_seed(seed + 2)
    W = torch.zeros(ld, device=dev)
    W[:game.d] = torch.randn(game.d, device=dev, generator=gen)
    E = torch.zeros(M, ld, device=dev)
    WX = torch.zeros(M, ld, device=dev)
    G = torch.zeros(M, ld, device=dev)
    wire = plan.new_wire(dev)
    n0 = float(torch.linalg.vector_norm(W[:game.d]))
    # w_{-1/2} = w_0 and e_0 = 0: the first evaluation points are
    # w_0 - (eta g_0 + e_0), the library's OMD step with q-hat = 0 (w stays w_0)
    G[:, :game.d] = game.operator(W[:game.d].expand(M, -1)) + noise * torch.randn(M, game.d, device=dev,
                                                                                   generator=gen)
    Q0 = torch.zeros(ld, device=dev)
    dqgan.omd_step(plan, eta, Q0, W, G, E, WX)
    del Q0
    hist = []
    for t in range(1, T + 1):
        G[:, :game.d] = game.operator(WX) + noise * torch.randn(M, game.d, device=dev, generator=gen)
        if on_step is not None:
            on_step(t, {"G": G, "E": E, "W": W, "plan": plan, "wire": wire, "WX": WX})
        dqgan.step_fused(plan, eta, t, G, E, W, WX, wire)
        if t % record_every == 0:
            hist.append(float(torch.linalg.vector_norm(W[:game.d])) / n0)
    plan.close()
    return hist


def run_gradient_descent(n=512, T=800, eta=0.2, seed=0):
    """Plain simultaneous gradient steps on the same game (no extrapolation,
    no compression): ||z_T|| / ||z_0||."""
    dev = torch.device("cuda")
    game = BilinearGame(n, seed, dev)
    gen = torch.Generator(device=dev).manual_seed(seed + 2)
    z = torch.randn(1, game.d, device=dev, generator=gen)
    n0 = float(torch.linalg.vector_norm(z))
    for _ in range(T):
        z = z - eta * game.operator(z)
    return float(torch.linalg.vector_norm(z)) / n0
