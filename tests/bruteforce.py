"""Independent dense fp64 reference for tiny GASLoC problems (tests only).

Built from library routines and the paper's matrix form, not from the
oracle's loops:
  * inner loop: one torch.optim.AdamW per worker (persistent state),
    App. B "Optimization";
  * outer step: one torch.optim.SGD per worker fed the negated pseudo-gradient
    x_t - x_{t,H} (Eq. 1 outer loop; Nesterov per section 4), which leaves
    the post-outer iterate z = x + eta*g (mu = 0) in the parameter;
  * mixing and consensus momentum: the matrix form of Eq. 2,
    x_{t+1} = W z_t + gamma (z_t - z_{t-1}) for t >= 1, as a dense matmul.
"""
import numpy as np
import torch


def laplacian(n, edges, weights):
    """Lambda = 1/2 sum_{(i,j)} lambda_ij (e_i - e_j)(e_i - e_j)^T (section 3.1, Notation)."""
    L = np.zeros((n, n))
    for (a, b), lam in zip(edges, weights):
        e = np.zeros(n)
        e[a] += 1.0
        e[b] -= 1.0
        L += 0.5 * lam * np.outer(e, e)
    return L


def run_rounds(x0, grads, W_of_round, H_i, rounds, lr, beta1, beta2, eps, wd, eta, mu, nesterov, gamma):
    """Return (x, y, u, z_prev, ce_list) after `rounds` rounds, all fp64.

    x0          [n, P] initial replicas
    grads(s)    fp64 [n, P] gradients of global local-step s
    W_of_round  t -> dense [n, n] mixing matrix
    H_i         local steps per worker
    """
    n, P = x0.shape
    x = x0.astype(np.float64).copy()
    inner = [torch.nn.Parameter(torch.zeros(P, dtype=torch.float64)) for _ in range(n)]
    outer = [torch.nn.Parameter(torch.tensor(x[i])) for i in range(n)]
    adam = [torch.optim.AdamW([inner[i]], lr=lr, betas=(beta1, beta2), eps=eps, weight_decay=wd)
            for i in range(n)]
    sgd = [torch.optim.SGD([outer[i]], lr=eta, momentum=mu, nesterov=nesterov and mu > 0)
           for i in range(n)]
    z_prev = None
    ces = []
    step = 0
    H_i = np.asarray(H_i)
    y = x.copy()
    for t in range(rounds):
        with torch.no_grad():
            for i in range(n):
                inner[i].copy_(torch.from_numpy(x[i]))
        for h in range(int(H_i.max())):
            g = grads(step)
            step += 1
            for i in range(n):
                if H_i[i] > h:
                    inner[i].grad = torch.from_numpy(np.ascontiguousarray(g[i], dtype=np.float64))
                    adam[i].step()
        y = np.stack([inner[i].detach().numpy().copy() for i in range(n)])
        z = np.empty_like(x)
        for i in range(n):
            with torch.no_grad():
                outer[i].copy_(torch.from_numpy(x[i]))
            outer[i].grad = torch.from_numpy(x[i] - y[i])
            sgd[i].step()
            z[i] = outer[i].detach().numpy()
        W = W_of_round(t)
        x_new = W @ z
        if gamma != 0.0 and t >= 1:
            x_new = x_new + gamma * (z - z_prev)
        z_prev = z
        x = x_new
        xbar = x.mean(axis=0)
        ces.append(float(((x - xbar) ** 2).sum()))
    u = np.stack([sgd[i].state[outer[i]]["momentum_buffer"].numpy().copy()
                  if mu > 0 else np.zeros(P) for i in range(n)])
    return x, y, u, z_prev, ces
